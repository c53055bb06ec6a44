// Spatial order of the two clouds for the dense scans.
//
// Every pair whose distance can matter to a row or a column lies within a
// small radius (the kept ball of Sec. III-B, Eq. 1, or the second minimum of
// Sec. III-A). With each cloud sorted along a Hilbert curve, a run of 32
// consecutive points occupies a small box, and the dense scans skip every
// run whose box is provably beyond that radius from the box of their rows
// (dense.hip). The order only decides which work is skipped: results do not
// depend on it.
//
//   k_spatial_sort  one workgroup per (sample, cloud, chunk of 8192 points).
//                   The frame is the bounding cube of both clouds of the
//                   sample, quantized to 10 bits per axis; the upper 20 bits of the 30-bit Hilbert keys are sorted by a
//                   least-significant-digit radix sort (two 10-bit digits,
//                   stable: ranks within a wave from ballots, across waves
//                   from per-wave digit counts in LDS). The sorted points are
//                   written as (x, y, z, original index), with the bounding
//                   box of every run of 32.
//   k_sort_merge    larger clouds: the sorted chunks merged pairwise, one
//                   level per launch (merge-path splits, 16 outputs per
//                   thread), then k_sort_gather writes the points and boxes.
#include <algorithm>

#include "apml_internal.h"
#include "device_common.h"

namespace apml {
namespace {

constexpr int kSortT = 1024;
constexpr int kSortWaves = kSortT / 64;
constexpr int kDigitBits = 10;
constexpr int kBins = 1 << kDigitBits; // == kSortT: one bin per thread in the scans
constexpr int kPasses = 3;
constexpr int kFirstPass = 1; // the lowest digit is not sorted (see k_spatial_sort)
constexpr int kSuper = 8; // keys per thread held in registers between global round trips
// Points sorted by one workgroup. A larger cloud is sorted in chunks of this
// many points in parallel, and the chunks are then merged pairwise.
constexpr int kSortChunk = kSuper * kSortT;
static_assert(kSortChunk == kSortChunkPoints, "chunk size");
constexpr int kMergeK = 16; // outputs per thread of a merge
static_assert(kBins == kSortT, "one bin per thread");

// Spreads the low 10 bits of v to every third bit (bit k goes to bit 3k).
__device__ __forceinline__ uint32_t spread3(uint32_t v)
{
    v &= 0x3FFu;
    v = (v | (v << 16)) & 0x030000FFu;
    v = (v | (v << 8)) & 0x0300F00Fu;
    v = (v | (v << 4)) & 0x030C30C3u;
    v = (v | (v << 2)) & 0x09249249u;
    return v;
}

// Position along the Hilbert curve of the cell (x, y, z), 10 bits per axis,
// by Skilling's transposition ("Programming the Hilbert curve", 2004): the
// axes are turned into the transposed Hilbert index, whose bits interleaved
// give the 30-bit key. Consecutive keys are adjacent cells, so a run of
// consecutive points stays compact (a Morton order jumps across the space).
__device__ __forceinline__ uint32_t hilbert_key(uint32_t x, uint32_t y, uint32_t z)
{
    uint32_t X[3] = {x, y, z};
#pragma unroll
    for (uint32_t Q = 1u << 9; Q > 1; Q >>= 1) {
        const uint32_t P = Q - 1;
#pragma unroll
        for (int i = 0; i < 3; ++i) {
            if (X[i] & Q) {
                X[0] ^= P; // invert the low bits of the first axis
            } else {       // exchange the low bits of the first axis and axis i
                const uint32_t t = (X[0] ^ X[i]) & P;
                X[0] ^= t;
                X[i] ^= t;
            }
        }
    }
    X[1] ^= X[0]; // Gray encode
    X[2] ^= X[1];
    uint32_t t = 0;
#pragma unroll
    for (uint32_t Q = 1u << 9; Q > 1; Q >>= 1)
        if (X[2] & Q)
            t ^= Q - 1;
    X[0] ^= t;
    X[1] ^= t;
    X[2] ^= t;
    return spread3(X[2]) | spread3(X[1]) << 1 | spread3(X[0]) << 2;
}

__device__ __forceinline__ uint32_t quantize(float v, float lo, float scale)
{
    const float t = (v - lo) * scale;
    return (uint32_t)fminf(fmaxf(t, 0.0f), 1023.0f);
}

// LDS of k_spatial_sort (dynamic; about 140 KB).
struct SortLds {
    int whist[kSortWaves][kBins]; // digit counts of each wave in the current tile (zero outside a tile)
    int woff[kSortWaves][kBins];  // their exclusive prefix over the waves
    int base[kPasses][kBins];     // next output position of every digit, per pass
    float frame[kSortWaves][6];
    int wsum[kSortWaves];
};

__device__ __forceinline__ uint64_t lanes_below() { return (1ull << lane_id()) - 1ull; }

// One stable pass: the n keys and values of src, in order of digit pass p.
__device__ void radix_pass(SortLds &s, int p, int n, const uint32_t *sk, const uint32_t *sv, uint32_t *dk,
                           uint32_t *dv)
{
    const int tid = threadIdx.x, wave = tid >> 6;
    const int shift = p * kDigitBits;
    for (int t0 = 0; t0 < n; t0 += kSuper * kSortT) {
        uint32_t key[kSuper], val[kSuper];
#pragma unroll
        for (int u = 0; u < kSuper; ++u) { // one global round trip for kSuper tiles
            const int k = t0 + u * kSortT + tid;
            key[u] = k < n ? sk[k] : 0u;
            val[u] = k < n ? sv[k] : 0u;
        }
#pragma unroll
        for (int u = 0; u < kSuper; ++u) {
            const int k0 = t0 + u * kSortT;
            if (k0 >= n) // uniform over the workgroup
                break;
            const bool valid = k0 + tid < n;
            const uint32_t dg = (key[u] >> shift) & (kBins - 1);
            uint64_t peers = __ballot(valid);
#pragma unroll
            for (int i = 0; i < kDigitBits; ++i) {
                const uint64_t bal = __ballot((dg >> i) & 1u);
                peers &= ((dg >> i) & 1u) ? bal : ~bal;
            }
            const uint64_t lower = peers & lanes_below();
            const int rank = __popcll(lower);
            const bool leader = valid && lower == 0;
            if (leader)
                s.whist[wave][dg] = __popcll(peers);
            lds_barrier();
            int run = 0;
#pragma unroll
            for (int w = 0; w < kSortWaves; ++w) {
                const int c = s.whist[w][tid];
                s.woff[w][tid] = run;
                run += c;
            }
            lds_barrier();
            const int pos = s.base[p][dg] + s.woff[wave][dg] + rank;
            if (valid && pos < n) { // always below n: every pass sees the digits the histograms counted
                dk[pos] = key[u];
                dv[pos] = val[u];
            }
            lds_barrier();
            s.base[p][tid] += run;
            if (leader) // this wave's next tile writes its counts after these clears (same wave, in order)
                s.whist[wave][dg] = 0;
        }
    }
}

// Bounding box of points [k0, k1) of sample b, numbered over X then Y, into
// f (min x, y, z, max x, y, z; every thread of the workgroup gets it). wf:
// LDS for the per-wave boxes. Ends with an LDS barrier.
__device__ void frame_of(const SpatialArgs &a, int b, int k0, int k1, float f[6], float (*wf)[6])
{
    const int tid = threadIdx.x, lane = lane_id(), wave = tid >> 6;
    const float *xs = a.x + (size_t)b * a.N * 3, *ys = a.y + (size_t)b * a.M * 3;
#pragma unroll
    for (int c = 0; c < 3; ++c) {
        f[c] = kInf;
        f[3 + c] = -kInf;
    }
    for (int k = k0 + tid; k < k1; k += kSortT) {
        const float *p = k < a.N ? xs + 3 * (size_t)k : ys + 3 * (size_t)(k - a.N);
#pragma unroll
        for (int c = 0; c < 3; ++c) {
            f[c] = fminf(f[c], p[c]);
            f[3 + c] = fmaxf(f[3 + c], p[c]);
        }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1)
#pragma unroll
        for (int c = 0; c < 3; ++c) {
            f[c] = fminf(f[c], __shfl_xor(f[c], o));
            f[3 + c] = fmaxf(f[3 + c], __shfl_xor(f[3 + c], o));
        }
    if (lane == 0)
#pragma unroll
        for (int c = 0; c < 6; ++c)
            wf[wave][c] = f[c];
    lds_barrier();
#pragma unroll
    for (int w = 0; w < kSortWaves; ++w)
#pragma unroll
        for (int c = 0; c < 3; ++c) {
            f[c] = fminf(f[c], wf[w][c]);
            f[3 + c] = fmaxf(f[3 + c], wf[w][3 + c]);
        }
}

// Clouds sorted in chunks: the partial boxes of slice blockIdx.y of sample
// blockIdx.x (both clouds), combined by every chunk of the sample.
__global__ __launch_bounds__(kSortT) void k_sort_frame(SpatialArgs a)
{
    __shared__ float wf[kSortWaves][6];
    const int b = blockIdx.x, q = blockIdx.y, n = a.N + a.M;
    const int per = (n + a.frame_slices - 1) / a.frame_slices;
    float f[6];
    frame_of(a, b, q * per, min(n, (q + 1) * per), f, wf);
    if (threadIdx.x < 6)
        a.frame_part[((size_t)b * a.frame_slices + q) * 6 + threadIdx.x] = f[threadIdx.x];
}

__global__ __launch_bounds__(kSortT) void k_spatial_sort(SpatialArgs a)
{
    extern __shared__ int4 lds_raw[];
    SortLds &s = *reinterpret_cast<SortLds *>(lds_raw);
    // workgroup: (sample, cloud, chunk of kSortChunk points)
    const int chunks = (max(a.N, a.M) + kSortChunk - 1) / kSortChunk;
    const int c = blockIdx.x % chunks, b = blockIdx.x / chunks / 2, cloud = blockIdx.x / chunks % 2;
    const int tid = threadIdx.x, lane = lane_id(), wave = tid >> 6;
    if (blockIdx.x == 0 && tid < 2 * kScanSlots) {
        (&a.ctr->scanned[0][0])[tid] = 0;
        if (tid == 0) {
            a.ctr->error = 0;
            a.ctr->overflow = 0;
        }
    }
    const int n_all = cloud ? a.M : a.N;
    const int c0 = c * kSortChunk;
    if (c0 >= n_all) // this cloud has fewer chunks (uniform over the workgroup)
        return;
    const int n = min(kSortChunk, n_all - c0);
    const int pad = cloud ? a.pad_y : a.pad_x;
    const float *pts_all = (cloud ? a.y : a.x) + (size_t)b * n_all * 3;
    const float *pts = pts_all + (size_t)c0 * 3;
    const size_t seg = (cloud ? (size_t)a.B * a.pad_x + (size_t)b * a.pad_y : (size_t)b * a.pad_x) + c0;
    uint32_t *k0 = a.key[0] + seg, *v0 = a.val[0] + seg, *k1 = a.key[1] + seg, *v1 = a.val[1] + seg;

    // frame: bounding cube of both clouds of the sample (from the partial
    // cubes of k_sort_frame when the clouds are sorted in chunks)
    float f[6];
    if (a.frame_part)
#pragma unroll
        for (int c = 0; c < 6; ++c) {
            f[c] = c < 3 ? kInf : -kInf;
            for (int q = 0; q < a.frame_slices; ++q) {
                const float v = a.frame_part[((size_t)b * a.frame_slices + q) * 6 + c];
                f[c] = c < 3 ? fminf(f[c], v) : fmaxf(f[c], v);
            }
        }
    else
        frame_of(a, b, 0, a.N + a.M, f, s.frame);
    for (int i = tid; i < kPasses * kBins; i += kSortT)
        (&s.base[0][0])[i] = 0;
    for (int i = tid; i < kSortWaves * kBins; i += kSortT)
        (&s.whist[0][0])[i] = 0;
    lds_barrier();
    const float ext = fmaxf(fmaxf(f[3] - f[0], f[4] - f[1]), f[5] - f[2]);
    const float scale = ext > 0.0f ? 1024.0f / ext : 0.0f;

    // keys and the digit histograms of the passes (independent of the order).
    // Only the upper 20 of the key's 30 bits are sorted (the lowest digit is
    // cleared, so the merges of larger clouds compare the same keys): 2^20
    // cells hold runs of 32 points about as compact as 2^30 for the clouds
    // sorted here, and one radix pass fewer is needed. The order only decides
    // which pairs the scans skip, never a result.
    for (int k = tid; k < n; k += kSortT) {
        const float *p = pts + 3 * (size_t)k;
        const uint32_t key =
            hilbert_key(quantize(p[0], f[0], scale), quantize(p[1], f[1], scale), quantize(p[2], f[2], scale)) &
            ~(uint32_t)(kBins - 1);
        k1[k] = key;
        v1[k] = (uint32_t)(c0 + k); // index within the sample
#pragma unroll
        for (int q = kFirstPass; q < kPasses; ++q)
            atomicAdd(&s.base[q][(key >> (q * kDigitBits)) & (kBins - 1)], 1);
    }
    __syncthreads(); // the keys written above are read back by other threads
    // exclusive scans of the histograms: bin tid of every pass
#pragma unroll
    for (int q = kFirstPass; q < kPasses; ++q) {
        const int c = s.base[q][tid];
        int inc = c;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const int v = __shfl_up(inc, o);
            if (lane >= o)
                inc += v;
        }
        if (lane == 63)
            s.wsum[wave] = inc;
        lds_barrier();
        int before = 0;
#pragma unroll
        for (int w = 0; w < kSortWaves; ++w)
            before += w < wave ? s.wsum[w] : 0;
        lds_barrier();
        s.base[q][tid] = before + inc - c;
    }
    lds_barrier();
    static_assert(kPasses - kFirstPass == 2, "two passes: from the second buffers back to them");
    radix_pass(s, 1, n, k1, v1, k0, v0);
    __syncthreads();
    radix_pass(s, 2, n, k0, v0, k1, v1);
    if (chunks > 1) // merged, then written out, by the next launches
        return;
    __syncthreads();

    // sorted points and the boxes of the runs of 32 (padding: empty boxes)
    float4 *out = (cloud ? a.sy : a.sx) + (size_t)b * pad;
    Box *box = (cloud ? a.box_y : a.box_x) + (size_t)b * (pad / kRun);
    for (int k = tid; k < pad; k += kSortT) { // pad is a multiple of 64: whole waves
        float4 v = make_float4(0.0f, 0.0f, 0.0f, __int_as_float(-1));
        float lo[3] = {kInf, kInf, kInf}, hi[3] = {-kInf, -kInf, -kInf};
        if (k < n) {
            const uint32_t i = v1[k];
            const float *p = pts_all + 3 * (size_t)i;
            v = make_float4(p[0], p[1], p[2], __uint_as_float(i));
            lo[0] = hi[0] = p[0];
            lo[1] = hi[1] = p[1];
            lo[2] = hi[2] = p[2];
        }
        out[k] = v;
#pragma unroll
        for (int o = 1; o < kRun; o <<= 1)
#pragma unroll
            for (int c = 0; c < 3; ++c) {
                lo[c] = fminf(lo[c], __shfl_xor(lo[c], o));
                hi[c] = fmaxf(hi[c], __shfl_xor(hi[c], o));
            }
        if ((lane & (kRun - 1)) == 0)
            box[k / kRun] = Box{make_float4(lo[0], lo[1], lo[2], 0.0f), make_float4(hi[0], hi[1], hi[2], 0.0f)};
    }
}

// One level of the pairwise merge of sorted runs of length run (key and value
// arrays src -> 1 - src), in every (sample, cloud) segment: thread t of a
// segment writes outputs kMergeK t ... kMergeK t + kMergeK - 1. Its start in
// each of the two runs comes from a binary search along the merge path
// (ties: the first run first).
__global__ __launch_bounds__(kBlock) void k_sort_merge(SpatialArgs a, int run, int src)
{
    const int64_t g = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    const int64_t per_x = (a.pad_x + kMergeK - 1) / kMergeK, per_y = (a.pad_y + kMergeK - 1) / kMergeK;
    const int64_t nx = (int64_t)a.B * per_x;
    const int cloud = g < nx ? 0 : 1;
    const int64_t h = cloud ? g - nx : g;
    const int64_t per = cloud ? per_y : per_x;
    if (h >= (int64_t)a.B * per)
        return;
    const int b = (int)(h / per), k0 = (int)(h - (int64_t)b * per) * kMergeK;
    const int n = cloud ? a.M : a.N;
    if (k0 >= n)
        return;
    const size_t seg = cloud ? (size_t)a.B * a.pad_x + (size_t)b * a.pad_y : (size_t)b * a.pad_x;
    const uint32_t *sk = a.key[src] + seg, *sv = a.val[src] + seg;
    uint32_t *dk = a.key[1 - src] + seg, *dv = a.val[1 - src] + seg;
    const int p0 = k0 / (2 * run) * (2 * run);        // the pair of runs holding output k0
    const int la = min(run, n - p0), lb = max(0, min(run, n - p0 - run));
    const uint32_t *A = sk + p0, *Bk = sk + p0 + la;
    const int d = k0 - p0;
    int lo = max(0, d - lb), hi = min(d, la);
    while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (A[mid] <= Bk[d - 1 - mid])
            lo = mid + 1;
        else
            hi = mid;
    }
    int i = lo, j = d - lo;
    const int end = min(p0 + la + lb, k0 + kMergeK);
    for (int k = k0; k < end; ++k) {
        const bool from_a = j >= lb || (i < la && A[i] <= Bk[j]);
        const int q = from_a ? p0 + i : p0 + la + j;
        dk[k] = sk[q];
        dv[k] = sv[q];
        i += from_a ? 1 : 0;
        j += from_a ? 0 : 1;
    }
}

// The sorted points (x, y, z, index in the sample) and the boxes of the runs
// of 32 from the final values (array src), one thread per output position.
__global__ __launch_bounds__(kBlock) void k_sort_gather(SpatialArgs a, int src)
{
    const int64_t g = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    const int64_t nx = (int64_t)a.B * a.pad_x;
    const int cloud = g < nx ? 0 : 1;
    const int64_t h = cloud ? g - nx : g;
    const int pad = cloud ? a.pad_y : a.pad_x;
    if (h >= (int64_t)a.B * pad) // whole waves: pad and nx are multiples of 64
        return;
    const int b = (int)(h / pad), k = (int)(h - (int64_t)b * pad);
    const int n = cloud ? a.M : a.N;
    const size_t seg = cloud ? (size_t)a.B * a.pad_x + (size_t)b * a.pad_y : (size_t)b * a.pad_x;
    const float *pts = (cloud ? a.y : a.x) + (size_t)b * n * 3;
    float4 v = make_float4(0.0f, 0.0f, 0.0f, __int_as_float(-1));
    float lo[3] = {kInf, kInf, kInf}, hi[3] = {-kInf, -kInf, -kInf};
    if (k < n) {
        const uint32_t i = a.val[src][seg + k];
        const float *p = pts + 3 * (size_t)i;
        v = make_float4(p[0], p[1], p[2], __uint_as_float(i));
        lo[0] = hi[0] = p[0];
        lo[1] = hi[1] = p[1];
        lo[2] = hi[2] = p[2];
    }
    (cloud ? a.sy : a.sx)[(size_t)b * pad + k] = v;
#pragma unroll
    for (int o = 1; o < kRun; o <<= 1)
#pragma unroll
        for (int c = 0; c < 3; ++c) {
            lo[c] = fminf(lo[c], __shfl_xor(lo[c], o));
            hi[c] = fmaxf(hi[c], __shfl_xor(hi[c], o));
        }
    if ((lane_id() & (kRun - 1)) == 0)
        (cloud ? a.box_y : a.box_x)[((size_t)b * pad + k) / kRun] =
            Box{make_float4(lo[0], lo[1], lo[2], 0.0f), make_float4(hi[0], hi[1], hi[2], 0.0f)};
}

// Box of each batch of 64 runs: one wave per (cloud, sample, batch), one lane
// per run (coalesced loads), then wave-wide min / max.
__global__ __launch_bounds__(kBlock) void k_batch_boxes(const Box *box_x, const Box *box_y, Box *batch_x,
                                                        Box *batch_y, int B, int pad_x, int pad_y, bool columns_only)
{
    const int64_t g = ((int64_t)blockIdx.x * kBlock + threadIdx.x) >> 6;
    const int lane = lane_id();
    const int nbx = batches(pad_x), nby = batches(pad_y);
    const int64_t nx = columns_only ? 0 : (int64_t)B * nbx;
    const int cloud = g < nx ? 0 : 1;
    const int64_t h = cloud ? g - nx : g;
    const int nbt = cloud ? nby : nbx, pad = cloud ? pad_y : pad_x;
    if (h >= (int64_t)B * nbt) // the whole wave
        return;
    const int b = (int)(h / nbt), t = (int)(h - (int64_t)b * nbt);
    const int runs = pad / kRun, r = t * 64 + lane;
    const Box *rb = (cloud ? box_y : box_x) + (size_t)b * runs;
    float4 lo = make_float4(kInf, kInf, kInf, 0.0f), hi = make_float4(-kInf, -kInf, -kInf, -kInf);
    if (r < runs) {
        lo = rb[r].lo;
        hi = rb[r].hi;
    }
    for (int off = 32; off > 0; off >>= 1) {
        lo.x = fminf(lo.x, __shfl_xor(lo.x, off));
        lo.y = fminf(lo.y, __shfl_xor(lo.y, off));
        lo.z = fminf(lo.z, __shfl_xor(lo.z, off));
        hi.x = fmaxf(hi.x, __shfl_xor(hi.x, off));
        hi.y = fmaxf(hi.y, __shfl_xor(hi.y, off));
        hi.z = fmaxf(hi.z, __shfl_xor(hi.z, off));
        hi.w = fmaxf(hi.w, __shfl_xor(hi.w, off));
    }
    if (lane == 0)
        (cloud ? batch_y : batch_x)[(size_t)b * nbt + t] = Box{make_float4(lo.x, lo.y, lo.z, 0.0f), hi};
}

} // namespace

size_t spatial_sort_lds() { return sizeof(SortLds); }

void launch_batch_boxes(const Box *box_x, const Box *box_y, Box *batch_x, Box *batch_y, int B, int pad_x, int pad_y,
                        bool columns_only, hipStream_t s)
{
    const int64_t n = (int64_t)B * ((columns_only ? 0 : batches(pad_x)) + batches(pad_y));
    hipLaunchKernelGGL(k_batch_boxes, dim3(blocks_for(64 * n, kBlock)), dim3(kBlock), 0, s, box_x, box_y, batch_x,
                       batch_y, B, pad_x, pad_y, columns_only);
}

hipError_t launch_spatial_sort(const SpatialArgs &a, hipStream_t s)
{
    const hipError_t e = set_dynamic_lds((const void *)k_spatial_sort, sizeof(SortLds));
    if (e != hipSuccess)
        return e;
    const int n_max = std::max(a.N, a.M);
    const int chunks = (n_max + kSortChunk - 1) / kSortChunk;
    if (a.frame_part)
        hipLaunchKernelGGL(k_sort_frame, dim3(a.B, a.frame_slices), dim3(kSortT), 0, s, a);
    hipLaunchKernelGGL(k_spatial_sort, dim3(2 * a.B * chunks), dim3(kSortT), sizeof(SortLds), s, a);
    if (chunks > 1) { // merge the sorted chunks pairwise, then write the points out
        int src = 1; // the radix sort ends in the second buffers
        const int64_t threads = (int64_t)a.B * ((a.pad_x + kMergeK - 1) / kMergeK + (a.pad_y + kMergeK - 1) / kMergeK);
        for (int run = kSortChunk; run < n_max; run *= 2, src = 1 - src)
            hipLaunchKernelGGL(k_sort_merge, dim3(blocks_for(threads, kBlock)), dim3(kBlock), 0, s, a, run, src);
        hipLaunchKernelGGL(k_sort_gather, dim3(blocks_for((int64_t)a.B * (a.pad_x + a.pad_y), kBlock)), dim3(kBlock),
                           0, s, a, src);
    }
    return hipGetLastError();
}

} // namespace apml
