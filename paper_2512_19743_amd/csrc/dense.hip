// Dense phase of the sparse APML loss: the two scans over all B*N*M pairs.
// VALU-bound; no matrix cores (the K=3 contraction is not a GEMM).
//
//   k_top2_pairs  per row and per column, the minimum and second minimum of
//              the single-precision squared distance (Sec. III-A), each pair
//              evaluated once: a lane holds eight rows, the columns stream
//              through scalar registers (wave-uniform loads), and a pair costs
//              6 VALU ops for the distance, 2 (min, med3) for its row's
//              statistics and 2 for its column's, whose per-lane partials
//              are merged across the wave once per eight columns.
//   k_finalize merges the per-chunk statistics and derives each row's and
//              column's emission threshold: the kept set s >= tau is the ball
//              C <= C1 + log(1/tau)/T (Sec. III-B, Eq. 1), widened by a small
//              relative margin and never below the second minimum.
//   k_emit     the candidate support: every pair inside its row's or its
//              column's threshold. Per pair 6 VALU ops for the distance, a max
//              of the two radii, a compare and an add-with-carry that records
//              the hit in a per-lane bitmask of 32 columns. A first pass counts
//              the hits per (row, column chunk) and per column and keeps them
//              (the first few of every (row, chunk) in its slots, the rest of
//              a tile in a pool region); once the offsets are known, a
//              compaction writes each row's pairs, in column order, into the
//              CSR arrays. Only tiles whose hits did not fit are scanned a
//              second time. The exact test s >= tau is applied later in
//              double precision on this candidate set.
#include <algorithm>
#include <utility>

#include "apml_internal.h"
#include "device_common.h"
#include "pieces.h"

namespace apml {
namespace {

// ---------------------------------------------------------------------------
// the minimum scan with one evaluation per pair
// ---------------------------------------------------------------------------
//
// A workgroup takes 64 kPairR rows of a sample, held by each of its waves
// (kPairR per lane), and one chunk of columns, a quarter per wave, which a
// wave streams through scalar registers in batches of eight, as the support
// scan streams them; the waves' row statistics are merged in LDS at the end. A pair costs the six operations
// of its distance, two for its row's statistics (in the lane's registers)
// and two for its column's statistics over the lane's rows, against 16 when
// rows and columns are scanned separately. After each batch the eight
// columns' statistics are merged across the 64 lanes: lane halves swap
// columns (v_permlane32_swap, then v_permlane16_swap) so that each merge step
// also halves the columns a lane holds, then 8-lane halves of each DPP row
// exchange their last two columns and a butterfly finishes: about 54
// operations per batch, under one per pair. Both statistics are
// order-independent (minimum and second minimum of the multiset; the merge
// of two top-2 multisets is exact), so the values are those of separate row
// and column scans, bit for bit. Rows past N sit at +inf and columns past
// the chunk at -inf: every pair involving one has distance +inf, which
// changes no statistic of a real point.

// The top-2 multiset (a1 <= a2) merged with (b1 <= b2): the second smallest
// of the four is med3(a1, b1, min(a2, b2)). Minima written out: the compiler
// would first canonicalize operands that come from lane permutations.
__device__ __forceinline__ void top2_merge(float &a1, float &a2, float b1, float b2)
{
    float m;
    asm("v_min_f32 %0, %1, %2" : "=v"(m) : "v"(a2), "v"(b2));
    a2 = __builtin_amdgcn_fmed3f(a1, b1, m);
    asm("v_min_f32 %0, %1, %2" : "=v"(a1) : "v"(a1), "v"(b1));
}

template <int CTRL> __device__ __forceinline__ float dpp_mov(float v)
{
    return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), CTRL, 0xF, 0xF, true));
}

// Lane swaps between two registers, for both statistics: v_permlane32_swap
// exchanges lanes 32-63 of the first register with lanes 0-31 of the second,
// v_permlane16_swap the odd 16-lane rows of the first with the even rows of
// the second. Written out: this compiler's builtins for them returned the
// first register's new value for both results once those fed further
// arithmetic (the merged statistics came out wrong), which inline assembly
// avoids; the waits around them are kept by hand.
__device__ __forceinline__ void swap32(float &a1, float &b1, float &a2, float &b2)
{
    asm volatile("s_nop 1\n\tv_permlane32_swap_b32 %0, %1\n\tv_permlane32_swap_b32 %2, %3\n\ts_nop 1"
                 : "+v"(a1), "+v"(b1), "+v"(a2), "+v"(b2));
}
__device__ __forceinline__ void swap16(float &a1, float &b1, float &a2, float &b2)
{
    asm volatile("s_nop 1\n\tv_permlane16_swap_b32 %0, %1\n\tv_permlane16_swap_b32 %2, %3\n\ts_nop 1"
                 : "+v"(a1), "+v"(b1), "+v"(a2), "+v"(b2));
}

// Merges the eight columns' statistics (c1[u], c2[u]) of all 64 lanes; on
// return lane 16 r (r = 0..3) holds column 2 r and lane 16 r + 8 column
// 2 r + 1 of the batch.
__device__ __forceinline__ void batch_merge(float (&c1)[8], float (&c2)[8], float &o1, float &o2)
{
    // lanes 0-31 keep columns 0-3, lanes 32-63 columns 4-7
    float d1[4], d2[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        float y1 = c1[k + 4], y2 = c2[k + 4];
        d1[k] = c1[k];
        d2[k] = c2[k];
        swap32(d1[k], y1, d2[k], y2);
        top2_merge(d1[k], d2[k], y1, y2);
    }
    // 16-lane row r of d[k] holds column k + 4 (r / 2); after the swap of odd
    // rows of d[k] with even rows of d[k + 2], row r holds column k + 2 r
    float e1[2], e2[2];
#pragma unroll
    for (int k = 0; k < 2; ++k) {
        float y1 = d1[k + 2], y2 = d2[k + 2];
        e1[k] = d1[k];
        e2[k] = d2[k];
        swap16(e1[k], y1, e2[k], y2);
        top2_merge(e1[k], e2[k], y1, y2);
    }
    // lanes 0-7 of each row keep e[0] (column 2 r), lanes 8-15 e[1] (2 r + 1);
    // each sends the other to the lane 8 places away (row_ror:8)
    const bool hi = (threadIdx.x & 8u) != 0;
    float k1 = hi ? e1[1] : e1[0], k2 = hi ? e2[1] : e2[0];
    top2_merge(k1, k2, dpp_mov<0x128>(hi ? e1[0] : e1[1]), dpp_mov<0x128>(hi ? e2[0] : e2[1]));
    // butterfly over the eight lanes: xor 1, xor 2 (quad_perm), then the
    // mirror within 8 (every lane of a quad then holds the same values)
    top2_merge(k1, k2, dpp_mov<0xB1>(k1), dpp_mov<0xB1>(k2));
    top2_merge(k1, k2, dpp_mov<0x4E>(k1), dpp_mov<0x4E>(k2));
    top2_merge(k1, k2, dpp_mov<0x141>(k1), dpp_mov<0x141>(k2));
    o1 = k1;
    o2 = k2;
}

// One batch of eight columns from j (scalar loads) against the lane's rows:
// the rows' statistics, and the columns' statistics merged over the wave
// and stored by lanes 16 r and 16 r + 8. TAIL: columns from cend on are
// placed at -inf (not loaded).
template <bool TAIL>
__device__ __forceinline__ void pair_batch(const float (&ax)[kPairR], const float (&ay)[kPairR],
                                           const float (&az)[kPairR], float (&m1)[kPairR], float (&m2)[kPairR],
                                           const_ptr<float> q, int j, int cend, float2 *colp)
{
    float c1[8], c2[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
        const int jj = TAIL ? min(j + u, cend - 1) : j + u;
        float bx = q[3 * jj], by = q[3 * jj + 1], bz = q[3 * jj + 2];
        if (TAIL && j + u >= cend) // wave-uniform
            bx = by = bz = -kInf;
        c1[u] = c2[u] = kInf;
#pragma unroll
        for (int v = 0; v < kPairR; ++v) {
            const float s = sqdist_f32(ax[v], ay[v], az[v], bx, by, bz);
            m2[v] = __builtin_amdgcn_fmed3f(m1[v], m2[v], s);
            m1[v] = fminf(m1[v], s);
            c2[u] = __builtin_amdgcn_fmed3f(c1[u], c2[u], s);
            c1[u] = fminf(c1[u], s);
        }
    }
    float o1, o2;
    batch_merge(c1, c2, o1, o2);
    const int lane = threadIdx.x & 63;
    if ((lane & 7) == 0) {
        const int col = j + 2 * (lane >> 4) + ((lane >> 3) & 1);
        if (!TAIL || col < cend)
            colp[col] = make_float2(o1, o2);
    }
}

__global__ __launch_bounds__(kPairThreads, 4) void k_top2_pairs(PairScan a)
{
    __shared__ float2 rows[kPairWaves][64 * kPairR]; // the waves' row statistics, merged at the end
    int t = blockIdx.x;
    const int cb = t % a.S_r;
    t /= a.S_r;
    const int rblk = t % a.S_c, b = t / a.S_c;
    const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
    // the workgroup's 64 kPairR rows, lane l holding rows l, l + 64, ... in
    // every wave; wave w takes the w-th quarter of the workgroup's columns
    float ax[kPairR], ay[kPairR], az[kPairR], m1[kPairR], m2[kPairR];
    const int rbase = rblk * 64 * kPairR;
#pragma unroll
    for (int v = 0; v < kPairR; ++v) {
        const int i = rbase + v * 64 + lane;
        if (i < a.N) {
            const float *p = a.x + ((size_t)b * a.N + i) * 3;
            ax[v] = p[0];
            ay[v] = p[1];
            az[v] = p[2];
        } else {
            ax[v] = ay[v] = az[v] = kInf;
        }
        m1[v] = m2[v] = kInf;
    }
    const int sub = a.chunk / kPairWaves;
    const int c0 = cb * a.chunk + w * sub, cend = min(a.M, c0 + sub);
    const const_ptr<float> q = as_const(a.y + (size_t)b * a.M * 3);
    float2 *colp = a.col_partial + ((size_t)rblk * a.B + b) * a.M;
    int j = c0;
    for (; j + 8 <= cend; j += 8)
        pair_batch<false>(ax, ay, az, m1, m2, q, j, cend, colp);
    if (j < cend)
        pair_batch<true>(ax, ay, az, m1, m2, q, j, cend, colp);
#pragma unroll
    for (int v = 0; v < kPairR; ++v)
        rows[w][v * 64 + lane] = make_float2(m1[v], m2[v]);
    __syncthreads();
    for (int k = threadIdx.x; k < 64 * kPairR; k += kPairThreads) {
        const int i = rbase + k;
        if (i >= a.N)
            break;
        float r1 = kInf, r2 = kInf;
#pragma unroll
        for (int u = 0; u < kPairWaves; ++u) { // top-2 of the union of the waves' top-2 multisets
            const float2 e = rows[u][k];
            r2 = fminf(fmaxf(r1, e.x), fminf(r2, e.y));
            r1 = fminf(r1, e.x);
        }
        a.row_partial[(size_t)cb * a.B * a.N + (size_t)b * a.N + i] = make_float2(r1, r2);
    }
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
        args.ctr->spill_fill = 0;
    }
    const int which = k < args.rows ? 0 : 1;
    if (which)
        k -= args.rows;
    const FinalizeDir &d = args.dir[which];
    if (k >= args.B * d.n_own)
        return;
    const size_t stride = (size_t)args.B * d.n_own;
    // the top-2 of a union of multisets does not depend on the order of the
    // merges: the chunks' partials are loaded kFinBatch at a time, so their
    // loads are in flight together
    constexpr int kFinBatch = 8;
    float m1 = kInf, m2 = kInf;
    for (int c0 = 0; c0 < d.S; c0 += kFinBatch) {
        float2 v[kFinBatch];
#pragma unroll
        for (int u = 0; u < kFinBatch; ++u)
            v[u] = c0 + u < d.S ? d.partial[(size_t)(c0 + u) * stride + k] : make_float2(kInf, kInf);
#pragma unroll
        for (int u = 0; u < kFinBatch; ++u) { // top-2 of the union of two top-2 multisets
            m2 = fminf(fmaxf(m1, v[u].x), fminf(m2, v[u].y));
            m1 = fminf(m1, v[u].x);
        }
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
    __shared__ uint2 list[kTileList]; // further hits: row in the tile << 16 | offset, rank in the row's
    __shared__ int row_start[kBlock], wave_sum[kBlock / 64], n_list, base_sh;
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
        if (threadIdx.x == 0)
            n_list = 0;
        __syncthreads();
        int cnt = 0;
        for_each_hit(ax, ay, az, E, q, j0, j1, keep, [&](int j) {
            atomicAdd(&col_cnt[j], 1);
            if (stage) {
                if (cnt < a.kst) {
                    stage_put(a, slot, cnt, j - j0);
                } else {
                    const int k = atomicAdd(&n_list, 1);
                    if (k < kTileList)
                        list[k] = make_uint2((uint32_t)threadIdx.x << 16 | (uint32_t)(j - j0), cnt - a.kst);
                }
            }
            ++cnt;
        });
        if (valid)
            a.cnt[slot] = cnt;
        const int extra = max(cnt - a.kst, 0);
        if (stage && !__syncthreads_or(extra > 0)) { // every hit of the tile in its slots
            if (threadIdx.x == 0)
                a.spill_base[t] = 0;
        } else if (stage) {
            // the rows' starts in the tile's region: an exclusive scan of
            // their further hits over the workgroup
            const int lane = lane_id(), wave = threadIdx.x >> 6;
            int incl = extra;
            for (int o = 1; o < 64; o <<= 1) {
                const int v = __shfl_up(incl, o);
                if (lane >= o)
                    incl += v;
            }
            if (lane == 63)
                wave_sum[wave] = incl;
            __syncthreads();
            int before = 0, total = 0;
#pragma unroll
            for (int w = 0; w < kBlock / 64; ++w) {
                before += w < wave ? wave_sum[w] : 0;
                total += wave_sum[w];
            }
            row_start[threadIdx.x] = before + incl - extra;
            if (threadIdx.x == 0) {
                int base = total == 0 ? 0 : -1;
                if (total > 0 && total <= kTileList) {
                    const int64_t need = kBlock + total;
                    const int64_t got = (int64_t)atomicAdd(&a.ctr->spill_fill, (unsigned long long)need);
                    if (got + need <= a.spill_cap)
                        base = (int)got;
                }
                if (base < 0)
                    atomicOr(&a.ctr->overflow, 1u);
                a.spill_base[t] = base;
                base_sh = base;
            }
            __syncthreads();
            const int base = base_sh;
            if (total > 0 && base >= 0) {
                uint16_t *reg = a.spill + base;
                reg[threadIdx.x] = (uint16_t)row_start[threadIdx.x];
                for (int u = threadIdx.x; u < total; u += kBlock) {
                    const uint2 e = list[u];
                    reg[kBlock + row_start[e.x >> 16] + (int)e.y] = (uint16_t)(e.x & 0xFFFFu);
                }
            }
        }
    } else {
        if (a.stage && a.spill_base[t] >= 0) // rescan only the tiles whose further hits did not fit
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
// kst come from the row's part of its tile's pool region (increasing column). With
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
    const int base = a.spill_base[t];
    if (base < 0) // the writing pass rescans this tile
        return;
    const int j0 = ch * a.chunk, gc0 = b * a.M + j0;
    const int ns = min(n, a.kst);
#pragma unroll
    for (int k = 0; k < kStage; ++k) // fixed trip count: the pairs' loads and atomics overlap
        if (k < ns) {
            const int jj = stage_get(a, (size_t)g, k);
            emit_pair<PLACE>(a, pos + k, row, i, gc0 + jj, j0 + jj);
        }
    if (n > a.kst) { // the row's further hits, in increasing column, from the tile's region
        const uint16_t *reg = a.spill + base;
        const uint16_t *mine = reg + kBlock + reg[i % kBlock];
        for (int k = a.kst; k < n; ++k) {
            const int jj = mine[k - a.kst];
            emit_pair<PLACE>(a, pos + k, row, i, gc0 + jj, j0 + jj);
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

void choose_pair_scan(PairScan &p, int B, int N, int M)
{
    // about kPairTargetWaves waves; each workgroup's chunk a multiple of 32
    // columns (eight per wave and batch), at most kPairMaxChunk
    p.B = B;
    p.N = N;
    p.M = M;
    p.S_c = (N + 64 * kPairR - 1) / (64 * kPairR);
    const int64_t blocks = (int64_t)B * p.S_c;
    const int unit = 8 * kPairWaves, units = (M + unit - 1) / unit;
    int64_t s = std::max<int64_t>(1, (kPairTargetWaves / kPairWaves + blocks - 1) / blocks);
    s = std::max<int64_t>(s, (units + kPairMaxChunk / unit - 1) / (kPairMaxChunk / unit));
    s = std::min<int64_t>(s, units);
    p.chunk = (int)((units + s - 1) / s) * unit;
    p.S_r = (M + p.chunk - 1) / p.chunk;
}

void launch_top2_pairs(const PairScan &p, hipStream_t s)
{
    hipLaunchKernelGGL(k_top2_pairs, dim3((unsigned)((int64_t)p.B * p.S_c * p.S_r)), dim3(kPairThreads), 0, s, p);
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
