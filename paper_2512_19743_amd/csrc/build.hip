// Sparse structure of the stored pairs: row-major order (CSR; each row's
// pairs in increasing column, written by the support scan) and a
// column-major permutation (CSC; each column's pairs in increasing row).
// The paper symmetrizes by concatenating the two COO streams and sorting
// 64-bit keys (Sec. III-C); here every pair is emitted once, with both
// memberships decided later, so only the column-major view needs building.
#include <algorithm>

#include "apml_internal.h"
#include "device_common.h"

namespace apml {
namespace {

// ---------------------------------------------------------------------------
// per-sample offsets
// ---------------------------------------------------------------------------

constexpr int kOffT = 1024;

// Pair count of owner k of sample b: the sum of a row's chunk counts (in
// 16-byte loads when the count is a multiple of 4), or a column's count.
__device__ __forceinline__ int owner_len(bool rows, const int32_t *cnt, int S, const int32_t *col_cnt, int b, int N,
                                         int M, int k)
{
    if (!rows)
        return col_cnt[(size_t)b * M + k];
    const int32_t *rc = cnt + ((size_t)b * N + k) * S;
    int len = 0, c = 0;
    if (S % 4 == 0)
        for (; c < S; c += 4) {
            const int4 v = *reinterpret_cast<const int4 *>(rc + c);
            len += v.x + v.y + v.z + v.w;
        }
    for (; c < S; ++c)
        len += rc[c];
    return len;
}

// Owners are cut into tiles of kOffTile; a workgroup of kOffT threads takes
// one tile of one sample and direction (grid: tiles x B x 2, blockIdx.z 0 for
// rows, 1 for columns), thread t owners tile * kOffTile + u * kOffT + t.
constexpr int kOffPer = 8;
constexpr int kOffTile = kOffT * kOffPer;

// Per tile: the pair total, the lane positions of its owners' piece groups and
// the largest piece count, into tiles[((dir * B + b) * T + tile) * 3 + 0..2].
__global__ __launch_bounds__(kOffT) void k_sample_scan(const int32_t *cnt, int S, const int32_t *col_cnt, int N,
                                                       int M, int32_t *tiles, int T)
{
    __shared__ int red[3][kOffT / 64];
    const int tile = blockIdx.x, b = blockIdx.y, B = gridDim.y, tid = threadIdx.x;
    const bool rows = blockIdx.z == 0;
    const int n = rows ? N : M;
    if (tile * kOffTile >= n) // the whole workgroup
        return;
    const int lane = lane_id(), wave = tid >> 6;
    int len[kOffPer];
#pragma unroll
    for (int u = 0; u < kOffPer; ++u) {
        const int k = tile * kOffTile + u * kOffT + tid;
        len[u] = k < n ? owner_len(rows, cnt, S, col_cnt, b, N, M, k) : -1;
    }
    int sum = 0, pos = 0, mx = 0;
#pragma unroll
    for (int u = 0; u < kOffPer; ++u)
        if (len[u] >= 0) {
            const int np = sink_pieces(len[u]);
            sum += len[u];
            pos += 1 << min(sink_log2_group(np), 30);
            mx = max(mx, np);
        }
    for (int off = 32; off > 0; off >>= 1) {
        sum += __shfl_xor(sum, off);
        pos += __shfl_xor(pos, off);
        mx = max(mx, __shfl_xor(mx, off));
    }
    if (lane == 0) {
        red[0][wave] = sum;
        red[1][wave] = pos;
        red[2][wave] = mx;
    }
    __syncthreads();
    if (tid == 0) {
        int t = 0, a = 0, m = 0;
        for (int w = 0; w < kOffT / 64; ++w) {
            t += red[0][w];
            a += red[1][w];
            m = max(m, red[2][w]);
        }
        int32_t *o = tiles + (((size_t)(rows ? 0 : 1) * B + b) * T + tile) * 3;
        o[0] = t;
        o[1] = a;
        o[2] = m;
    }
}

// The offsets of one tile: the base of its sample (pairs of the earlier
// samples) and of its tile within the sample, plus the exclusive scan of its
// owners' counts (one workgroup scan per round u). The first tile of each
// sample also closes row_ptr / col_ptr and fills the read-back block (totals,
// offsets, piece counts; the counters from sample 0's row tile).
__global__ __launch_bounds__(kOffT) void k_sample_base(const int32_t *cnt, int S, const int32_t *col_cnt,
                                                       const Counters *ctr, int N, int M, int32_t *row_ptr,
                                                       int32_t *col_ptr, const int32_t *tiles, int T,
                                                       Readback *rb_host)
{
    __shared__ int wsum[kOffT / 64];
    __shared__ int base_s;
    const int tile = blockIdx.x, b = blockIdx.y, B = gridDim.y, tid = threadIdx.x;
    const bool rows = blockIdx.z == 0;
    const int n = rows ? N : M;
    if (tile * kOffTile >= n)
        return;
    const int lane = lane_id(), wave = tid >> 6;
    const int32_t *tl = tiles + (size_t)(rows ? 0 : 1) * B * T * 3;
    if (wave == 0) {
        // pairs before this tile: all tiles of the earlier samples, then the
        // earlier tiles of this one (tile entries of a direction are in
        // sample-major order)
        const int before = b * T + tile, nt = (n + kOffTile - 1) / kOffTile;
        int64_t base = 0;
        for (int e = lane; e < before; e += 64)
            if (e % T < nt) // this direction's tiles (the grid covers the longer one)
                base += tl[3 * e];
        for (int off = 32; off > 0; off >>= 1)
            base += __shfl_xor(base, off);
        if (lane == 0)
            base_s = (int)base; // the host rejects totals beyond int32 before using any offset
        if (tile == 0) {
            int64_t tot = 0;
            int a = 0, m = 0;
            for (int e = lane; e < nt; e += 64) {
                tot += tl[3 * ((size_t)b * T + e)];
                a += tl[3 * ((size_t)b * T + e) + 1];
                m = max(m, tl[3 * ((size_t)b * T + e) + 2]);
            }
            for (int off = 32; off > 0; off >>= 1) {
                tot += __shfl_xor(tot, off);
                a += __shfl_xor(a, off);
                m = max(m, __shfl_xor(m, off));
            }
            if (lane == 0) {
                readback_totals(rb_host)[(rows ? 0 : B) + b] = tot;
                int32_t *pc = readback_pieces(rb_host, B) + 4 * b;
                pc[rows ? 0 : 1] = a;
                pc[rows ? 2 : 3] = m;
                if (rows)
                    readback_offsets(rb_host, B)[b] = (int)base;
                if (b == B - 1) {
                    const int end = (int)(base + tot);
                    (rows ? row_ptr[(size_t)B * N] : col_ptr[(size_t)B * M]) = end;
                    if (rows)
                        readback_offsets(rb_host, B)[B] = end;
                }
            }
        }
    }
    if (tile == 0 && b == 0 && rows) // the counters, word by word over the workgroup
        for (int i = tid; i < (int)(sizeof(Counters) / 4); i += kOffT)
            reinterpret_cast<uint32_t *>(&rb_host->ctr)[i] = reinterpret_cast<const uint32_t *>(ctr)[i];
    int len[kOffPer];
#pragma unroll
    for (int u = 0; u < kOffPer; ++u) {
        const int k = tile * kOffTile + u * kOffT + tid;
        len[u] = k < n ? owner_len(rows, cnt, S, col_cnt, b, N, M, k) : 0;
    }
    __syncthreads(); // base_s
    int carry = base_s;
    int32_t *out = rows ? row_ptr + (size_t)b * N : col_ptr + (size_t)b * M;
    const int rounds = min(kOffPer, (n - tile * kOffTile + kOffT - 1) / kOffT); // rounds holding owners
#pragma unroll
    for (int u = 0; u < kOffPer; ++u) {
        if (u >= rounds) // the same for the whole workgroup
            break;
        int inc = len[u];
        for (int off = 1; off < 64; off <<= 1) {
            const int v = __shfl_up(inc, off);
            if (lane >= off)
                inc += v;
        }
        if (lane == 63)
            wsum[wave] = inc;
        __syncthreads();
        int before = 0, all = 0;
        for (int w = 0; w < kOffT / 64; ++w) {
            before += w < wave ? wsum[w] : 0;
            all += wsum[w];
        }
        __syncthreads();
        const int k = tile * kOffTile + u * kOffT + tid;
        if (k < n)
            out[k] = carry + before + inc - len[u];
        carry += all;
    }
}

} // namespace

size_t offsets_scratch_ints(int B, int N, int M)
{
    const int T = (std::max(N, M) + kOffTile - 1) / kOffTile;
    return 3 * 2 * (size_t)B * T;
}

namespace {

// ---------------------------------------------------------------------------
// column-major permutation
// ---------------------------------------------------------------------------

// Places every pair in its column segment; the order inside a segment
// depends on the atomics and is fixed by k_csc_sort.
__global__ __launch_bounds__(kBlock) void k_csc_fill(DevPlan d, BuildArgs a)
{
    const int64_t t = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (t >= d.nnz)
        return;
    const int r = d.csr_row[t];
    const int b = r / d.N;
    const int gc = b * d.M + d.csr_col[t];
    const int p = d.col_ptr[gc] + atomicAdd(&a.col_fill[gc], 1);
    a.tmp_row[p] = r - b * d.N;
    a.tmp_src[p] = (int32_t)t;
    d.csc_col[p] = gc;
}

// The same placement for the pairs of sample blockIdx.x / ranges whose column
// lies in its range blockIdx.x % ranges of C columns (dynamic LDS: C ints):
// each column's next free slot is kept in LDS, starting at its global offset,
// and taken by an LDS atomic. The workgroup reads all of the sample's pairs
// and places those of its columns.
constexpr int kFillT = 1024;
constexpr int kFillBatch = 8;

__global__ __launch_bounds__(kFillT) void k_csc_fill_lds(DevPlan d, BuildArgs a, int ranges, int C)
{
    extern __shared__ int next[];
    const int b = blockIdx.x / ranges, q = blockIdx.x % ranges;
    const int j0 = q * C, j1 = min(d.M, j0 + C);
    const size_t gb = (size_t)b * d.M;
    for (int j = j0 + (int)threadIdx.x; j < j1; j += kFillT)
        next[j - j0] = d.col_ptr[gb + j];
    __syncthreads();
    const int lo = d.row_ptr[(size_t)b * d.N], hi = d.row_ptr[(size_t)(b + 1) * d.N];
    // kFillBatch pairs per thread with their loads in flight together (the
    // rows too, although only the pairs of this range use them)
    for (int t0 = lo; t0 < hi; t0 += kFillBatch * kFillT) {
        int j[kFillBatch], r[kFillBatch];
#pragma unroll
        for (int u = 0; u < kFillBatch; ++u) {
            const int t = t0 + u * kFillT + (int)threadIdx.x;
            j[u] = t < hi ? d.csr_col[t] : -1;
            r[u] = t < hi ? d.csr_row[t] : 0;
        }
#pragma unroll
        for (int u = 0; u < kFillBatch; ++u)
            if (j[u] >= j0 && j[u] < j1) {
                const int t = t0 + u * kFillT + (int)threadIdx.x;
                const int p = atomicAdd(&next[j[u] - j0], 1);
                a.tmp_row[p] = r[u] - b * d.N;
                a.tmp_src[p] = t;
                d.csc_col[p] = (int32_t)(gb + j[u]);
            }
    }
}

// Canonical order inside each column (increasing row): the rank of an entry
// is the number of entries of its column with a smaller row.
__global__ __launch_bounds__(kBlock) void k_csc_sort(DevPlan d, BuildArgs a)
{
    const int64_t p = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (p >= d.nnz)
        return;
    const int gc = d.csc_col[p];
    const int s0 = d.col_ptr[gc], s1 = d.col_ptr[gc + 1];
    const int key = a.tmp_row[p];
    const int rank = count_below(a.tmp_row, s0, s1, key);
    d.csc_row[s0 + rank] = key;
    d.csc_perm[s0 + rank] = a.tmp_src[p];
}

// Kept pairs of one chunk of kCountChunk stored pairs of sample blockIdx.y
// (grid: chunks x samples), into out[sample * chunks + chunk].
constexpr int kCountChunk = 8192;

__global__ __launch_bounds__(kBlock) void k_count_support(const int32_t *row_ptr,
                                                          const uint8_t *flags, int N,
                                                          unsigned long long *out)
{
    __shared__ unsigned long long part[kBlock / 64];
    const int b = blockIdx.y;
    const int t0 = row_ptr[(size_t)b * N], t1 = row_ptr[(size_t)(b + 1) * N];
    const int c0 = t0 + (int)blockIdx.x * kCountChunk, c1 = min(t1, c0 + kCountChunk);
    unsigned long long n = 0;
    for (int t = c0 + threadIdx.x; t < c1; t += kBlock)
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
        out[(size_t)b * gridDim.x + blockIdx.x] = s;
    }
}

} // namespace

void launch_offsets(const int32_t *cnt, int S, const int32_t *col_cnt, const Counters *ctr, int B, int N, int M,
                    int32_t *row_ptr, int32_t *col_ptr, int32_t *tiles, Readback *rb_host, hipStream_t s)
{
    const int T = (std::max(N, M) + kOffTile - 1) / kOffTile;
    hipLaunchKernelGGL(k_sample_scan, dim3(T, B, 2), dim3(kOffT), 0, s, cnt, S, col_cnt, N, M, tiles, T);
    hipLaunchKernelGGL(k_sample_base, dim3(T, B, 2), dim3(kOffT), 0, s, cnt, S, col_cnt, ctr, N, M, row_ptr, col_ptr,
                       (const int32_t *)tiles, T, rb_host);
}

void launch_csc_build(const DevPlan &d, const BuildArgs &a, hipStream_t s)
{
    // d.col_ptr holds the scan of the column counts (launch_col_scan). With
    // enough samples, column ranges of each sample in LDS (each workgroup
    // reads the sample's pairs once); else one thread per pair and a global
    // atomic per pair (measured at 64 x 8192 x 8192: 107 us).
    const unsigned g = blocks_for(d.nnz, kBlock);
    const int ranges = std::min(16, std::max((d.M + 16383) / 16384, (512 + d.B - 1) / d.B));
    const int C = (d.M + ranges - 1) / ranges;
    if (d.B * ranges >= 256 && C <= 16384) {
        hipLaunchKernelGGL(k_csc_fill_lds, dim3(d.B * ranges), dim3(kFillT), (size_t)C * sizeof(int), s, d, a, ranges,
                           C);
    } else {
        hipLaunchKernelGGL(k_csc_fill, dim3(g), dim3(kBlock), 0, s, d, a);
    }
    hipLaunchKernelGGL(k_csc_sort, dim3(g), dim3(kBlock), 0, s, d, a);
}

void launch_csc_sort(const DevPlan &d, const BuildArgs &a, hipStream_t s)
{
    hipLaunchKernelGGL(k_csc_sort, dim3(blocks_for(d.nnz, kBlock)), dim3(kBlock), 0, s, d, a);
}

int count_support_chunks(int64_t max_pairs) { return (int)std::max<int64_t>(1, (max_pairs + kCountChunk - 1) / kCountChunk); }

void launch_count_support(const int32_t *row_ptr, const uint8_t *flags, int B, int N, int chunks,
                          unsigned long long *out, hipStream_t s)
{
    hipLaunchKernelGGL(k_count_support, dim3(chunks, B), dim3(kBlock), 0, s, row_ptr, flags, N, out);
}

} // namespace apml
