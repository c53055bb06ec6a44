// Dense phase of the sparse APML loss: the two scans over all B*N*M pairs.
// VALU-bound; no matrix cores (the K=3 contraction is not a GEMM).
//
//   k_top2     per row and per column, the minimum and second minimum of the
//              single-precision squared distance (Sec. III-A). Each lane owns
//              one point; the other cloud is streamed through scalar registers
//              (wave-uniform loads), so a pair costs 6 VALU ops for the
//              distance and 2 (min, med3) for the statistics.
//   k_finalize merges the per-chunk statistics and derives each row's and
//              column's emission threshold: the kept set s >= tau is the ball
//              C <= C1 + log(1/tau)/T (Sec. III-B, Eq. 1), widened by a small
//              relative margin and never below the second minimum.
//   k_emit     the candidate support: every pair inside its row's or its
//              column's threshold. Per pair 6 VALU ops for the distance, a max
//              of the two radii, a compare and an add-with-carry that records
//              the hit in a per-lane bitmask of 32 columns. A first pass counts
//              the hits per (row, column chunk) and per column; once the
//              offsets are known, a second pass writes each row's pairs, in
//              column order, straight into the CSR arrays. The exact test
//              s >= tau is applied later in double precision on this
//              candidate set.
#include "apml_internal.h"
#include "device_common.h"
#include "pieces.h"

namespace apml {
namespace {

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

struct FinalizeArgs {
    FinalizeDir dir[2];
    int B;
    int rows; // B * n_own of dir[0]
    Params p;
    Counters *ctr;
};

__global__ __launch_bounds__(kBlock) void k_finalize(FinalizeArgs args)
{
    int k = blockIdx.x * kBlock + threadIdx.x;
    if (k == 0) { // the full scans leave the skipping scans' counts unused
        args.ctr->error = 0;
        args.ctr->overflow = 0;
    }
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
    const double e = emission_radius2(m1, m2, d.log_ratio, args.p);
    const float E = isinf(e) ? kInf : __double2float_ru(e);
    if (which == 0) {
        d.E[k] = E;
    } else {
        const float *o = d.own + (size_t)k * 3;
        d.packed[k] = make_float4(o[0], o[1], o[2], E);
        d.zero_a[k] = 0;
        d.zero_b[k] = 0;
    }
}

// Radius test of one pair (inside the row's ball E or the column's ball w),
// shifted into bits: bits = 2*bits + hit. Three VALU instructions; the
// compiler's own max would first canonicalize the scalar operand, and its
// bit insertion takes two more.
__device__ __forceinline__ uint32_t shift_in_hit(uint32_t bits, float ax, float ay, float az, float E,
                                                 f32x4 yv)
{
    const float s = sqdist_f32(ax, ay, az, yv.x, yv.y, yv.z);
    float m;
    asm("v_max_f32 %1, %3, %4\n\t"
        "v_cmp_le_f32 vcc, %2, %1\n\t"
        "v_addc_co_u32 %0, vcc, %0, %0, vcc"
        : "+v"(bits), "=&v"(m)
        : "v"(s), "s"(yv.w), "v"(E)
        : "vcc");
    return bits;
}

// Calls f(j) for every column j in [j0, j1) whose pair with this lane's row
// passes the radius test, in increasing j. Blocks of 32 columns: one bit per
// column is shifted in as the columns pass (first column in the top bit),
// then the lane visits its hits. keep masks out lanes that have no row.
template <class F>
__device__ __forceinline__ void for_each_hit(float ax, float ay, float az, float E, const_ptr<f32x4> q, int j0,
                                             int j1, uint32_t keep, F f)
{
    int j = j0;
    for (; j + 32 <= j1; j += 32) {
        uint32_t bits = 0;
#pragma unroll
        for (int u = 0; u < 32; ++u)
            bits = shift_in_hit(bits, ax, ay, az, E, q[j + u]);
        bits &= keep;
        while (bits) {
            const int u = __clz(bits);
            f(j + u);
            bits &= ~(0x80000000u >> u);
        }
    }
    if (j < j1) {
        uint32_t bits = 0;
        const int n = j1 - j;
        for (int u = 0; u < n; ++u)
            bits = shift_in_hit(bits, ax, ay, az, E, q[j + u]);
        bits = (bits << (32 - n)) & keep;
        while (bits) {
            const int u = __clz(bits);
            f(j + u);
            bits &= ~(0x80000000u >> u);
        }
    }
}

// Staged hit k of (row, chunk) slot: the column's offset within the chunk,
// in one byte when every chunk has at most 256 columns, else in two.
__device__ __forceinline__ void stage_put(const EmitArgs &a, size_t slot, int k, int v)
{
    if (a.stage_narrow)
        reinterpret_cast<uint8_t *>(a.stage)[slot * a.kst + k] = (uint8_t)v;
    else
        a.stage[slot * a.kst + k] = (uint16_t)v;
}

__device__ __forceinline__ int stage_get(const EmitArgs &a, size_t slot, int k)
{
    return a.stage_narrow ? (int)reinterpret_cast<const uint8_t *>(a.stage)[slot * a.kst + k]
                          : (int)a.stage[slot * a.kst + k];
}

// Pass 1 (WRITE = false) counts the hits of each (row, chunk) and of each
// column; pass 2 writes them, in increasing column, at the row's CSR offset
// plus the counts of the row's earlier chunks. Both passes take bitwise the
// same decisions.
template <bool WRITE> __global__ __launch_bounds__(kBlock) void k_emit(EmitArgs a)
{
    __shared__ int n_spill;
    const int t = blockIdx.x;
    const int ob = t % a.owner_blocks;
    const int rest = t / a.owner_blocks;
    const int ch = rest % a.S;
    const int b = rest / a.S;
    const int i = ob * kBlock + threadIdx.x;
    const bool valid = i < a.N;
    const int row = b * a.N + (valid ? i : a.N - 1);
    const float *p = a.x + (size_t)row * 3;
    const float ax = p[0], ay = p[1], az = p[2];
    const float E = valid ? a.E_row[row] : -kInf;
    const_ptr<f32x4> q = as_const(reinterpret_cast<const f32x4 *>(a.ypack + (size_t)b * a.M));
    const int j0 = ch * a.chunk;
    const int j1 = min(a.M, j0 + a.chunk);
    const uint32_t keep = valid ? ~0u : 0u; // a lane without a row ignores the columns' balls too
    if (!WRITE) {
        int32_t *col_cnt = a.col_cnt + (size_t)b * a.M;
        const bool stage = a.stage != nullptr;
        const size_t slot = (size_t)row * a.S + ch;
        uint32_t *spill = a.stage ? a.spill + (size_t)t * kTileSpill : nullptr;
        if (threadIdx.x == 0)
            n_spill = 0;
        __syncthreads();
        int cnt = 0;
        for_each_hit(ax, ay, az, E, q, j0, j1, keep, [&](int j) {
            atomicAdd(&col_cnt[j], 1);
            if (stage) {
                if (cnt < a.kst) {
                    stage_put(a, slot, cnt, j - j0);
                } else { // in increasing j for each row
                    const int k = atomicAdd(&n_spill, 1);
                    if (k < kTileSpill)
                        spill[k] = (uint32_t)threadIdx.x << 16 | (uint32_t)(j - j0);
                }
            }
            ++cnt;
        });
        if (valid)
            a.cnt[(size_t)row * a.S + ch] = cnt;
        if (stage) {
            __syncthreads();
            if (threadIdx.x == 0) {
                a.spill_n[t] = n_spill;
                if (n_spill > kTileSpill)
                    atomicOr(&a.ctr->overflow, 1u);
            }
        }
    } else {
        if (a.stage && a.spill_n[t] <= kTileSpill) // rescan only the tiles whose list overflowed
            return;
        int pos = a.row_ptr[row];
        for (int c = 0; c < ch; ++c)
            pos += a.cnt[(size_t)row * a.S + c];
        for_each_hit(ax, ay, az, E, q, j0, j1, keep, [&](int j) {
            a.csr_col[pos] = j;
            a.csr_row[pos] = row;
            ++pos;
        });
    }
}

// CSR from the staged hits: one thread per (row, chunk) writes its hits at
// the row's offset plus the hits of the row's earlier chunks; hits beyond
// kst come from the tile list, in list order (increasing column). With
// PLACE, each pair also takes a slot in its column segment (k_csc_sort then
// fixes the order inside the segment).
template <bool PLACE>
__device__ __forceinline__ void emit_pair(const EmitArgs &a, int pos, int row, int i, int gc, int j)
{
    a.csr_col[pos] = j;
    a.csr_row[pos] = row;
    if (PLACE) {
        const int p = a.col_ptr[gc] + atomicAdd(&a.col_fill[gc], 1);
        a.tmp_row[p] = i;
        a.tmp_src[p] = pos;
        a.csc_col[p] = gc;
    }
}

template <bool PLACE> __device__ __forceinline__ void emit_compact_thread(const EmitArgs &a, int64_t g)
{
    if (g >= (int64_t)a.B * a.N * a.S)
        return;
    const int row = (int)(g / a.S), ch = (int)(g % a.S);
    const int b = row / a.N, i = row - b * a.N;
    const int t = (b * a.S + ch) * a.owner_blocks + i / kBlock; // the tile of the counting pass
    const int32_t *cnt = a.cnt + (size_t)row * a.S;
    int pos = a.row_ptr[row];
    for (int c = 0; c < ch; ++c)
        pos += cnt[c];
    const int n = cnt[ch];
    const int n_spill = a.spill_n[t];
    if (n_spill > kTileSpill) // the writing pass rescans this tile
        return;
    const int j0 = ch * a.chunk, gc0 = b * a.M + j0;
    const int ns = min(n, a.kst);
#pragma unroll
    for (int k = 0; k < kStage; ++k) // fixed trip count: the pairs' loads and atomics overlap
        if (k < ns) {
            const int jj = stage_get(a, (size_t)g, k);
            emit_pair<PLACE>(a, pos + k, row, i, gc0 + jj, j0 + jj);
        }
    if (n > a.kst) {
        const uint32_t *sp = a.spill + (size_t)t * kTileSpill;
        const uint32_t me = (uint32_t)(i % kBlock);
        int k = a.kst;
        for (int u = 0; u < n_spill; ++u)
            if (sp[u] >> 16 == me) {
                const int jj = (int)(sp[u] & 0xFFFFu);
                emit_pair<PLACE>(a, pos + k, row, i, gc0 + jj, j0 + jj);
                ++k;
            }
    }
}

template <bool PLACE> __global__ __launch_bounds__(kBlock) void k_emit_compact(EmitArgs a)
{
    emit_compact_thread<PLACE>(a, (int64_t)blockIdx.x * kBlock + threadIdx.x);
}

// The compaction (first n_compact blocks) and, in the remaining blocks, the
// placement of the per-sample Sinkhorn pieces (block k: sample k / 2, order
// k % 2): independent work in one launch, so the placement runs on the CUs
// the compaction leaves free.
constexpr int kFusedT = kSinkLanes;

__global__ __launch_bounds__(kFusedT) void k_emit_compact_place(EmitArgs a, DevPlan d, int32_t *place,
                                                                 int n_compact)
{
    __shared__ int hist[8], base[8];
    if ((int)blockIdx.x < n_compact) {
        emit_compact_thread<false>(a, (int64_t)blockIdx.x * kFusedT + threadIdx.x);
        return;
    }
    const int k = blockIdx.x - n_compact;
    pieces::place_order(d, place, k / 2, k % 2 == 0, hist, base);
}

} // namespace

void launch_top2(const ScanDir &rows, const ScanDir &cols, int B, hipStream_t s)
{
    Top2Args a{{rows, cols}, B};
    hipLaunchKernelGGL(k_top2, dim3(rows.tiles + cols.tiles), dim3(kBlock), 0, s, a);
}

void launch_finalize(const FinalizeDir &rows, const FinalizeDir &cols, int B, const Params &p,
                     Counters *ctr, hipStream_t s)
{
    FinalizeArgs a{{rows, cols}, B, B * rows.n_own, p, ctr};
    hipLaunchKernelGGL(k_finalize, dim3(blocks_for((int64_t)B * (rows.n_own + cols.n_own), kBlock)),
                       dim3(kBlock), 0, s, a);
}

void launch_emit_count(const EmitArgs &a, hipStream_t s)
{
    hipLaunchKernelGGL(k_emit<false>, dim3(a.B * a.S * a.owner_blocks), dim3(kBlock), 0, s, a);
}

void launch_emit_write(const EmitArgs &a, hipStream_t s)
{
    hipLaunchKernelGGL(k_emit<true>, dim3(a.B * a.S * a.owner_blocks), dim3(kBlock), 0, s, a);
}

void launch_emit_compact(const EmitArgs &a, bool overflow, bool place, const DevPlan *d, int32_t *pieces_place,
                         hipStream_t s)
{
    if (pieces_place && !place) { // with the placement of the Sinkhorn pieces in the same launch
        const int nc = (int)blocks_for((int64_t)a.B * a.N * a.S, kFusedT);
        hipLaunchKernelGGL(k_emit_compact_place, dim3(nc + 2 * a.B), dim3(kFusedT), 0, s, a, *d, pieces_place, nc);
    } else if (overflow || !place) { // the rescanned tiles are placed by k_csc_fill afterwards
        hipLaunchKernelGGL(k_emit_compact<false>, dim3(blocks_for((int64_t)a.B * a.N * a.S, kBlock)), dim3(kBlock), 0,
                           s, a);
    } else {
        hipLaunchKernelGGL(k_emit_compact<true>, dim3(blocks_for((int64_t)a.B * a.N * a.S, kBlock)), dim3(kBlock), 0,
                           s, a);
    }
    if (overflow)
        hipLaunchKernelGGL(k_emit<true>, dim3(a.B * a.S * a.owner_blocks), dim3(kBlock), 0, s, a);
}

} // namespace apml
