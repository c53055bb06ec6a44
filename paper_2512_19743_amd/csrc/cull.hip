// Dense phase of the sparse APML loss for large samples: the two scans over
// the pairs of every sample, skipping the pairs that provably cannot matter.
// VALU-bound; no matrix cores (the K=3 contraction is not a GEMM). Small
// samples take the full scans of dense.hip instead.
//
// Both clouds are sorted along a space-filling curve (spatial.hip), with the
// box of every run of 32 points. A wave takes 64 consecutive owners (one per
// lane) and streams the runs of the other cloud through scalar registers
// (wave-uniform loads), skipping every run whose box is farther from the
// owners' box than any distance that can still matter to them. The skip is
// exact: the squared gap between two boxes, evaluated with the same
// single-precision sequence as a pair's squared distance, never exceeds the
// value computed for any pair of points inside them (rounding is monotone),
// so a skipped pair would have been rejected by the very comparison the scan
// makes.
//
//   k_cull_top2     per row and per column, the minimum and second minimum of the
//              single-precision squared distance (Sec. III-A). A run is
//              skipped when its gap exceeds the current second minimum of
//              every owner of the wave: it cannot change either statistic.
//              The run at the owners' own place along the curve goes first,
//              then the batches of 64 runs in increasing gap and the runs of
//              each batch in increasing gap, so that the bound tightens as
//              early as possible.
//   k_cull_finalize back in the original order, each row's and column's emission
//              threshold: the kept set s >= tau is the ball
//              C <= C1 + log(1/tau)/T (Sec. III-B, Eq. 1), widened by a small
//              relative margin and never below the second minimum.
//   k_cull_emit     the candidate support: every pair inside its row's or its
//              column's threshold; a run is skipped when its gap exceeds both
//              the largest row threshold of the wave and the largest column
//              threshold of the run. Per pair 6 VALU ops for the distance, a
//              max of the two radii, a compare and an add-with-carry that
//              records the hit in a per-lane bitmask of the run. A first pass
//              counts the hits per row and per column; once the offsets are
//              known, a second pass writes each row's columns, and
//              k_cull_rank puts them in increasing column order. The exact
//              test s >= tau is applied later in double precision on this
//              candidate set.
#include "apml_internal.h"
#include "device_common.h"
#include "pieces.h"

namespace apml {
namespace {

constexpr int kWaves = kBlock / 64; // waves per workgroup of the scans
static_assert(kScanRows == 64, "one owner per lane");
static_assert(kWaves == 4, "four waves share the runs of 64 owners");

// Reductions over the 64 lanes of non-negative floats (or +inf / NaN), as
// unsigned bit patterns, which order them like the values. All lanes must be
// active (inactive lanes would contribute zeros): call them outside any
// condition, including the right operand of && or ||. Rows of 16 lanes by DPP,
// then the four rows through scalar registers.
__device__ __forceinline__ uint32_t row_max_u32(uint32_t v)
{
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xF, 0xF, false));  // quad_perm 1,0,3,2
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, false));  // quad_perm 2,3,0,1
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x141, 0xF, 0xF, false)); // row_half_mirror
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x140, 0xF, 0xF, false)); // row_mirror
    return v;
}

__device__ __forceinline__ uint32_t row_min_u32(uint32_t v)
{
    v = min(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xF, 0xF, false));
    v = min(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, false));
    v = min(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x141, 0xF, 0xF, false));
    v = min(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x140, 0xF, 0xF, false));
    return v;
}

__device__ __forceinline__ float wave_max_nonneg(float x)
{
    const uint32_t v = row_max_u32(__float_as_uint(x));
    const uint32_t a = max((uint32_t)__builtin_amdgcn_readlane(v, 0), (uint32_t)__builtin_amdgcn_readlane(v, 16));
    const uint32_t b = max((uint32_t)__builtin_amdgcn_readlane(v, 32), (uint32_t)__builtin_amdgcn_readlane(v, 48));
    return __uint_as_float(max(a, b));
}

__device__ __forceinline__ uint32_t wave_min_u32(uint32_t x)
{
    const uint32_t v = row_min_u32(x);
    const uint32_t a = min((uint32_t)__builtin_amdgcn_readlane(v, 0), (uint32_t)__builtin_amdgcn_readlane(v, 16));
    const uint32_t b = min((uint32_t)__builtin_amdgcn_readlane(v, 32), (uint32_t)__builtin_amdgcn_readlane(v, 48));
    return min(a, b);
}

// top-2 of the union of two top-2 multisets
__device__ __forceinline__ void merge_top2(float &m1, float &m2, float o1, float o2)
{
    m2 = fminf(fmaxf(m1, o1), fminf(m2, o2));
    m1 = fminf(m1, o1);
}

struct WaveBox {
    float lo[3], hi[3];
};

// Box of the wave's 64 owners: the union of their two runs (scalar loads).
__device__ __forceinline__ WaveBox owners_box(const Box *runs, int g, int n_own)
{
    const_ptr<f32x4> p = as_const(reinterpret_cast<const f32x4 *>(runs)); // lo, hi of run r at 2r, 2r + 1
    const f32x4 lo = p[4 * g], hi = p[4 * g + 1];
    WaveBox w{{lo.x, lo.y, lo.z}, {hi.x, hi.y, hi.z}};
    if ((2 * g + 1) * kRun < n_own) {
        const f32x4 lo2 = p[4 * g + 2], hi2 = p[4 * g + 3];
        w.lo[0] = fminf(w.lo[0], lo2.x);
        w.lo[1] = fminf(w.lo[1], lo2.y);
        w.lo[2] = fminf(w.lo[2], lo2.z);
        w.hi[0] = fmaxf(w.hi[0], hi2.x);
        w.hi[1] = fmaxf(w.hi[1], hi2.y);
        w.hi[2] = fmaxf(w.hi[2], hi2.z);
    }
    return w;
}

// Lower bound of the computed squared distance of any pair with one point in
// each box: the per-axis gaps through the same rounding sequence as
// sqdist_f32. For points a in the owners' box and p in box r,
// fl(p.x - a.x) >= fl(r.lo.x - hi.x) (and likewise on the other side), and
// squares and fused multiply-adds of non-negative values are monotone.
__device__ __forceinline__ float box_gap2(const WaveBox &w, const Box &r)
{
    const float gx = fmaxf(fmaxf(r.lo.x - w.hi[0], w.lo[0] - r.hi.x), 0.0f);
    const float gy = fmaxf(fmaxf(r.lo.y - w.hi[1], w.lo[1] - r.hi.y), 0.0f);
    const float gz = fmaxf(fmaxf(r.lo.z - w.hi[2], w.lo[2] - r.hi.z), 0.0f);
    return sqdist_f32(gx, gy, gz, 0.0f, 0.0f, 0.0f);
}

// The same bound for one point a and the box held by lane i (lo, hi in that
// lane's registers; i is wave-uniform, so the box arrives as scalars).
__device__ __forceinline__ float lane_box_gap2(float4 a, const float4 &lo, const float4 &hi, int i)
{
    auto bcast = [i](float v) { return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), i)); };
    const float gx = fmaxf(fmaxf(bcast(lo.x) - a.x, a.x - bcast(hi.x)), 0.0f);
    const float gy = fmaxf(fmaxf(bcast(lo.y) - a.y, a.y - bcast(hi.y)), 0.0f);
    const float gz = fmaxf(fmaxf(bcast(lo.z) - a.z, a.z - bcast(hi.z)), 0.0f);
    return sqdist_f32(gx, gy, gz, 0.0f, 0.0f, 0.0f);
}

__device__ __forceinline__ float box_gap2(const WaveBox &w, const float4 &lo, const float4 &hi)
{
    return box_gap2(w, Box{lo, hi});
}

struct Top2Args {
    CullDir dir[2];
    int B;
    int groups0; // B * dir[0].waves: workgroups of the first direction
    Counters *ctr;
};

// One workgroup per 64 owners; its kWaves waves take the runs r with
// r % kWaves == wave. Each wave publishes its owners' running (min, second
// min) in LDS after every run; a wave's skip bound merges its own with the
// other waves' latest values, which are always valid (they only decrease),
// so no synchronisation is needed until the final merge.
__global__ __launch_bounds__(kBlock) void k_cull_top2(Top2Args args)
{
    __shared__ float2 part[kWaves][kScanRows];
    int grp = xcd_contiguous(blockIdx.x, gridDim.x);
    const int which = grp < args.groups0 ? 0 : 1;
    if (which)
        grp -= args.groups0;
    const CullDir &d = args.dir[which];
    const int b = grp / d.waves, g = grp - b * d.waves;
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); // uniform to the compiler
    const int lane = lane_id();
    const int k = g * kScanRows + lane;
    const bool valid = k < d.n_own;
    const float4 a = d.own[(size_t)b * d.pad_own + min(k, d.n_own - 1)];
    const WaveBox wb = owners_box(d.own_box + (size_t)b * (d.pad_own / kRun), g, d.n_own);
    const_ptr<f32x4> bc = as_const(reinterpret_cast<const f32x4 *>(d.bc + (size_t)b * d.pad_bc));
    const Box *boxes = d.bc_box + (size_t)b * (d.pad_bc / kRun);
    const int nb = (d.n_bc + kRun - 1) / kRun;
    part[wv][lane] = make_float2(kInf, kInf);
    __syncthreads();
    volatile float2 *others = &part[0][lane];
    float m1 = kInf, m2 = kInf;
    int cols = 0;
    auto scan_run = [&](int r) { // r is wave-uniform: the run's points come through scalar loads
        const int j0 = r * kRun, n = min(kRun, d.n_bc - j0);
        if (n == kRun) {
#pragma unroll
            for (int u = 0; u < kRun; ++u) {
                const f32x4 v = bc[j0 + u];
                const float s = sqdist_f32(a.x, a.y, a.z, v.x, v.y, v.z);
                m2 = __builtin_amdgcn_fmed3f(m1, m2, s); // second order statistic of the multiset
                m1 = fminf(m1, s);
            }
        } else {
            for (int u = 0; u < n; ++u) {
                const f32x4 v = bc[j0 + u];
                const float s = sqdist_f32(a.x, a.y, a.z, v.x, v.y, v.z);
                m2 = __builtin_amdgcn_fmed3f(m1, m2, s);
                m1 = fminf(m1, s);
            }
        }
        cols += n;
        part[wv][lane] = make_float2(m1, m2);
    };
    // current second minimum of this lane's owner over the runs of all waves
    auto bound = [&]() {
        float b1 = m1, b2 = m2;
#pragma unroll
        for (int o = 0; o < kWaves; ++o) { // every entry read, this wave's own replaced (no branches)
            const float ox = others[o * kScanRows].x, oy = others[o * kScanRows].y;
            merge_top2(b1, b2, o == wv ? kInf : ox, o == wv ? kInf : oy);
        }
        return b2;
    };
    // the run at the owners' place along the curve first
    const int home = min(nb - 1, (int)(((int64_t)g * kScanRows + kScanRows / 2) * d.n_bc / d.n_own / kRun));
    if (home % kWaves == wv)
        scan_run(home);
    // Batches of 64 runs, 64 batches at a time (one per lane): the gaps of all
    // of them are formed at once, then the batches within the current bound
    // are visited nearest first. A batch beyond the bound costs one lane's
    // box test instead of a pass of the wave's loop.
    // The batch holding the home run goes first (its key 0; the others' keys
    // order them by gap).
    const int nbatch = (nb + 63) / 64;
    const Box *bboxes = d.bc_batch + (size_t)b * batches(d.pad_bc);
    for (int c0 = 0; c0 < nbatch; c0 += 64) {
        bool blive = c0 + lane < nbatch;
        float bgap = kInf;
        if (blive) {
            const Box bx = bboxes[c0 + lane];
            bgap = box_gap2(wb, bx.lo, bx.hi);
        }
        const uint32_t bkey = c0 + lane == home / 64 ? 0u : __float_as_uint(bgap) + 1u;
        for (;;) {
            // the largest current second minimum over the owners (a cross-lane
            // reduction: evaluated with every lane active, never under a condition)
            const float wave_bb = wave_max_nonneg(valid ? bound() : 0.0f);
            blive = blive && !(bgap > wave_bb);
            if (!__ballot(blive))
                break;
            const uint32_t bmin = wave_min_u32(blive ? bkey : 0xFFFFFFFFu);
            const int bi = __ffsll((unsigned long long)__ballot(blive && bkey == bmin)) - 1;
            blive = blive && lane != bi;
            const int base = (c0 + bi) * 64;
            const int r = base + lane;
            bool live = r < nb && r != home && r % kWaves == wv;
            float4 blo = make_float4(0.0f, 0.0f, 0.0f, 0.0f), bhi = blo;
            if (live) {
                blo = boxes[r].lo;
                bhi = boxes[r].hi;
            }
            const float gap = live ? box_gap2(wb, blo, bhi) : kInf;
            for (;;) {
                const float lb = bound();
                const float wave_lb = wave_max_nonneg(valid ? lb : 0.0f);
                live = live && !(gap > wave_lb);
                const uint64_t todo = __ballot(live);
                if (!todo)
                    break;
                // the nearest remaining run next
                const uint32_t gmin = wave_min_u32(live ? __float_as_uint(gap) : 0xFFFFFFFFu);
                const uint64_t pick = __ballot(live && __float_as_uint(gap) == gmin);
                const int i = __ffsll((unsigned long long)pick) - 1;
                live = live && lane != i;
                // and only if the run can matter to one of the owners themselves
                const float pg = lane_box_gap2(a, blo, bhi, i);
                if (__ballot(valid && !(pg > lb)))
                    scan_run(base + i);
            }
        }
    }
    __syncthreads();
    if (wv == 0) {
#pragma unroll
        for (int o = 1; o < kWaves; ++o) {
            const float2 v = part[o][lane];
            merge_top2(m1, m2, v.x, v.y);
        }
        if (valid)
            d.m12s[(size_t)b * d.pad_own + k] = make_float2(m1, m2);
    }
    if (lane == 0)
        atomicAdd(&args.ctr->scanned[0][blockIdx.x % kScanSlots],
                  (unsigned long long)cols * min(kScanRows, d.n_own - g * kScanRows));
}

struct FinalizeArgs {
    CullFinalizeDir dir[2];
    int B;
    int64_t split; // B * dir[0].pad
    Params p;
};

__global__ __launch_bounds__(kBlock) void k_cull_finalize(FinalizeArgs args)
{
    int64_t t = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    const int which = t < args.split ? 0 : 1;
    if (which)
        t -= args.split;
    const CullFinalizeDir &d = args.dir[which];
    if (t >= (int64_t)args.B * d.pad) // whole waves: pad and split are multiples of 64
        return;
    const int b = (int)(t / d.pad), k = (int)(t - (int64_t)b * d.pad);
    float E = -kInf;
    if (k < d.n_own) {
        const float4 o = d.own[t];
        const int i = __float_as_int(o.w);
        const float2 m = d.m12s[t];
        d.m12[(size_t)b * d.n_own + i] = m;
        const double e = emission_radius2(m.x, m.y, d.log_ratio, args.p);
        E = isinf(e) ? kInf : __double2float_ru(e);
        if (which == 0) {
            d.E[t] = E;
        } else {
            d.packed[t] = make_float4(o.x, o.y, o.z, E);
            d.zero_a[(size_t)b * d.n_own + i] = 0;
            d.zero_b[(size_t)b * d.n_own + i] = 0;
        }
    }
    if (which == 1) { // the largest threshold of every run of columns
#pragma unroll
        for (int o = 1; o < kRun; o <<= 1)
            E = fmaxf(E, __shfl_xor(E, o));
        if ((lane_id() & (kRun - 1)) == 0)
            d.box[t / kRun].hi.w = E;
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

// Pass 1 (WRITE = false) counts the hits of each row and of each column; pass
// 2 writes each row's columns (original indices) at the row's offset, in
// scan order. Both passes take bitwise the same decisions. One workgroup per
// 64 rows; its kWaves waves take the runs r with r % kWaves == wave.
template <bool WRITE> __global__ __launch_bounds__(kBlock) void k_cull_emit(CullEmitArgs a)
{
    __shared__ int acc[kWaves][kScanRows]; // per-wave counts (pass 1); fill of each row (pass 2)
    const int grp = xcd_contiguous(blockIdx.x, gridDim.x);
    const int b = grp / a.waves, g = grp - b * a.waves;
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); // uniform to the compiler
    const int lane = lane_id();
    const int k = g * kScanRows + lane;
    const bool valid = k < a.N;
    const float4 pa = a.sx[(size_t)b * a.pad_x + min(k, a.N - 1)];
    const int row = b * a.N + __float_as_int(pa.w);
    const float E = valid ? a.E[(size_t)b * a.pad_x + k] : -kInf;
    const WaveBox wb = owners_box(a.box_x + (size_t)b * (a.pad_x / kRun), g, a.N);
    const float wave_E = wave_max_nonneg(valid ? E : 0.0f);
    const_ptr<f32x4> yp = as_const(reinterpret_cast<const f32x4 *>(a.yp + (size_t)b * a.pad_y));
    const float4 *sy = a.sy + (size_t)b * a.pad_y;
    const Box *boxes = a.box_y + (size_t)b * (a.pad_y / kRun);
    const int nb = (a.M + kRun - 1) / kRun;
    int cols = 0;
    const int pos0 = valid && WRITE ? a.row_ptr[row] : 0;
    // pass 2 writes only the rows beyond the staging, in workgroups that have one
    if (WRITE && !a.wg_over[grp])
        return;
    const bool mine = WRITE ? valid && a.row_ptr[row + 1] - pos0 > kCullStage : valid;
    const uint32_t keep = mine ? ~0u : 0u; // a lane without a row ignores the columns' balls too
    if (wv == 0)
        acc[0][lane] = 0;
    __syncthreads();
    // the batches of 64 runs first, 64 of them at a time (one per lane); the
    // runs of the batches that can hold a hit then in increasing order
    const Box *bboxes = a.batch_y + (size_t)b * batches(a.pad_y);
    const int nbatch = (nb + 63) / 64;
    for (int c0 = 0; c0 < nbatch; c0 += 64) {
        bool reach = false;
        if (c0 + lane < nbatch) {
            const Box bx = bboxes[c0 + lane];
            reach = !(box_gap2(wb, bx.lo, bx.hi) > fmaxf(wave_E, bx.hi.w));
        }
        for (uint64_t btodo = __ballot(reach); btodo; btodo &= btodo - 1) {
            const int base = (c0 + __ffsll((unsigned long long)btodo) - 1) * 64;
            const int r = base + lane;
            bool take = false;
            float4 blo = make_float4(0.0f, 0.0f, 0.0f, 0.0f), bhi = blo;
            if (r < nb && r % kWaves == wv) {
                blo = boxes[r].lo;
                bhi = boxes[r].hi;
                take = !(box_gap2(wb, blo, bhi) > fmaxf(wave_E, bhi.w));
            }
            uint64_t todo = __ballot(take);
            while (todo) {
                const int rr = base + __ffsll((unsigned long long)todo) - 1;
                todo &= todo - 1;
                const int i = rr - base;
                const float run_E = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(bhi.w), i));
                const float gap = lane_box_gap2(pa, blo, bhi, i);
                if (!__ballot(valid && !(gap > fmaxf(E, run_E)))) // no row of the wave can reach the run
                    continue;
                const int j0 = rr * kRun, n = min(kRun, a.M - j0);
                // one bit per column, the run's first column in the top bit
                uint32_t bits = 0;
                if (n == kRun) {
#pragma unroll
                    for (int u = 0; u < kRun; ++u)
                        bits = shift_in_hit(bits, pa.x, pa.y, pa.z, E, yp[j0 + u]);
                } else {
                    for (int u = 0; u < n; ++u)
                        bits = shift_in_hit(bits, pa.x, pa.y, pa.z, E, yp[j0 + u]);
                    bits <<= kRun - n;
                }
                bits &= keep;
                cols += n;
                while (bits) {
                    const int u = __clz(bits);
                    bits &= ~(0x80000000u >> u);
                    const int j = __float_as_int(sy[j0 + u].w);
                    const int slot = atomicAdd(&acc[0][lane], 1); // this row's hits over the waves
                    if (WRITE) {
                        a.tmp_col[pos0 + slot] = j;
                        a.csr_row[pos0 + slot] = row;
                    } else {
                        if (slot < kCullStage)
                            a.stage[(size_t)row * kCullStage + slot] = j;
                        atomicAdd(&a.col_cnt[(size_t)b * a.M + j], 1);
                    }
                }
            }
        }
    }
    if (!WRITE) {
        __syncthreads();
        if (wv == 0) {
            const int n = acc[0][lane];
            if (valid)
                a.cnt[row] = n;
            if (__ballot(valid && n > kCullStage)) { // rare: pass 2 writes this workgroup's long rows
                if (lane == 0) {
                    a.wg_over[grp] = 1;
                    atomicOr(&a.ctr->overflow, 1u);
                }
            } else if (lane == 0) {
                a.wg_over[grp] = 0;
            }
        }
        if (lane == 0)
            atomicAdd(&a.ctr->scanned[1][blockIdx.x % kScanSlots],
                      (unsigned long long)cols * min(kScanRows, a.N - g * kScanRows));
    }
}

// Increasing column order inside a row that overflowed the staging: the
// rank of an entry is the number of entries of its row with a smaller column.
__device__ __forceinline__ void rank_entry(const CullEmitArgs &a, int64_t e)
{
    if (e >= a.nnz)
        return;
    const int r = a.csr_row[e];
    const int s0 = a.row_ptr[r], s1 = a.row_ptr[r + 1];
    if (s1 - s0 <= kCullStage) // ordered from the staging
        return;
    const int j = a.tmp_col[e];
    const int rank = count_below(a.tmp_col, s0, s1, j);
    a.csr_col[s0 + rank] = j;
}

__global__ __launch_bounds__(kBlock) void k_cull_rank(CullEmitArgs a)
{
    rank_entry(a, (int64_t)blockIdx.x * kBlock + threadIdx.x);
}

// Row r (global) from its staged columns, when they are all there: each goes
// to the position given by its rank among them.
__device__ __forceinline__ void order_row(const CullEmitArgs &a, int64_t r)
{
    if (r >= (int64_t)a.B * a.N)
        return;
    const int s0 = a.row_ptr[r], n = a.row_ptr[r + 1] - s0;
    if (n > kCullStage) // written and ranked by the overflow passes
        return;
    int j[kCullStage];
#pragma unroll
    for (int k = 0; k < kCullStage; ++k)
        j[k] = k < n ? a.stage[r * kCullStage + k] : INT_MAX;
#pragma unroll
    for (int k = 0; k < kCullStage; ++k) {
        int rank = 0;
#pragma unroll
        for (int q = 0; q < kCullStage; ++q)
            rank += j[q] < j[k];
        if (k < n) {
            a.csr_col[s0 + rank] = j[k];
            a.csr_row[s0 + k] = (int)r;
        }
    }
}

// The ordering (first n_rows blocks) and, in the remaining blocks, the
// placement of the per-sample Sinkhorn pieces (block k: sample k / 2, order
// k % 2): independent work in one launch, so the placement runs on the CUs
// the ordering leaves free.
constexpr int kFusedT = kSinkLanes;

__global__ __launch_bounds__(kFusedT) void k_cull_order_place(CullEmitArgs a, DevPlan d, int32_t *place, int n_rows)
{
    __shared__ int hist[8], base[8];
    if ((int)blockIdx.x < n_rows) {
        order_row(a, (int64_t)blockIdx.x * kFusedT + threadIdx.x);
        return;
    }
    const int k = blockIdx.x - n_rows;
    pieces::place_order(d, place, k / 2, k % 2 == 0, hist, base);
}

__global__ __launch_bounds__(kBlock) void k_cull_order(CullEmitArgs a)
{
    order_row(a, (int64_t)blockIdx.x * kBlock + threadIdx.x);
}

} // namespace

void launch_cull_top2(const CullDir &rows, const CullDir &cols, int B, Counters *ctr, hipStream_t s)
{
    Top2Args a{{rows, cols}, B, B * rows.waves, ctr};
    hipLaunchKernelGGL(k_cull_top2, dim3(B * (rows.waves + cols.waves)), dim3(kBlock), 0, s, a);
}

void launch_cull_finalize(const CullFinalizeDir &rows, const CullFinalizeDir &cols, int B, const Params &p,
                          hipStream_t s)
{
    FinalizeArgs a{{rows, cols}, B, (int64_t)B * rows.pad, p};
    hipLaunchKernelGGL(k_cull_finalize, dim3(blocks_for((int64_t)B * (rows.pad + cols.pad), kBlock)), dim3(kBlock), 0,
                       s, a);
}

void launch_cull_emit_count(const CullEmitArgs &a, hipStream_t s)
{
    hipLaunchKernelGGL(k_cull_emit<false>, dim3(a.B * a.waves), dim3(kBlock), 0, s, a);
}

void launch_cull_emit_write(const CullEmitArgs &a, hipStream_t s)
{
    hipLaunchKernelGGL(k_cull_emit<true>, dim3(a.B * a.waves), dim3(kBlock), 0, s, a);
}

void launch_cull_emit_order(const CullEmitArgs &a, const DevPlan *d, int32_t *pieces_place, hipStream_t s)
{
    const int64_t rows = (int64_t)a.B * a.N;
    if (pieces_place) {
        const int nr = (int)blocks_for(rows, kFusedT);
        hipLaunchKernelGGL(k_cull_order_place, dim3(nr + 2 * a.B), dim3(kFusedT), 0, s, a, *d, pieces_place, nr);
    } else {
        hipLaunchKernelGGL(k_cull_order, dim3(blocks_for(rows, kBlock)), dim3(kBlock), 0, s, a);
    }
}

void launch_cull_emit_rank(const CullEmitArgs &a, hipStream_t s)
{
    hipLaunchKernelGGL(k_cull_rank, dim3(blocks_for(a.nnz, kBlock)), dim3(kBlock), 0, s, a);
}

} // namespace apml
