// Sparse structure of the stored pairs: row-major order (CSR; each row's
// pairs in increasing column, written by the support scan) and a
// column-major permutation (CSC; each column's pairs in increasing row).
// The paper symmetrizes by concatenating the two COO streams and sorting
// 64-bit keys (Sec. III-C); here every pair is emitted once, with both
// memberships decided later, so only the column-major view needs building.
#include "apml_internal.h"
#include "device_common.h"

namespace apml {
namespace {

// ---------------------------------------------------------------------------
// exclusive prefix sums (three phases: tile sums, scan of tile sums, apply)
// ---------------------------------------------------------------------------

constexpr int kScanItems = 8;
constexpr int kScanTile = kBlock * kScanItems;

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

__global__ __launch_bounds__(kBlock) void k_scan_reduce(ScanArray a)
{
    const int k0 = blockIdx.x * kScanTile + threadIdx.x * kScanItems;
    int s = 0;
    for (int u = 0; u < kScanItems; ++u)
        s += scan_load(a, k0 + u);
    int total;
    block_exclusive_scan(s, &total);
    if (threadIdx.x == 0)
        a.tile_sums[blockIdx.x] = total;
}

__global__ __launch_bounds__(kBlock) void k_scan_tiles(ScanArray a)
{
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

__global__ __launch_bounds__(kBlock) void k_scan_apply(ScanArray a)
{
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
    int rank = 0;
    for (int q = s0; q < s1; ++q)
        rank += a.tmp_row[q] < key;
    d.csc_row[s0 + rank] = key;
    d.csc_perm[s0 + rank] = a.tmp_src[p];
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

} // namespace

int scan_tile_items() { return kScanTile; }

void launch_scan(const ScanArray &a, hipStream_t s)
{
    hipLaunchKernelGGL(k_scan_reduce, dim3(a.tiles), dim3(kBlock), 0, s, a);
    hipLaunchKernelGGL(k_scan_tiles, dim3(1), dim3(kBlock), 0, s, a);
    hipLaunchKernelGGL(k_scan_apply, dim3(a.tiles), dim3(kBlock), 0, s, a);
}


void launch_col_scan(const int32_t *col_cnt, int n, int32_t *col_ptr, int32_t *tiles, hipStream_t s)
{
    ScanArray sc{col_cnt, n, 1, col_ptr, tiles, (n + kScanTile - 1) / kScanTile};
    launch_scan(sc, s);
}

void launch_csc_build(const DevPlan &d, const BuildArgs &a, hipStream_t s)
{
    // d.col_ptr holds the scan of the column counts (launch_col_scan)
    const unsigned g = blocks_for(d.nnz, kBlock);
    hipLaunchKernelGGL(k_csc_fill, dim3(g), dim3(kBlock), 0, s, d, a);
    hipLaunchKernelGGL(k_csc_sort, dim3(g), dim3(kBlock), 0, s, d, a);
}

void launch_count_support(const int32_t *row_ptr, const uint8_t *flags, int B, int N,
                          unsigned long long *out, hipStream_t s)
{
    hipLaunchKernelGGL(k_count_support, dim3(B), dim3(kBlock), 0, s, row_ptr, flags, N, out);
}

} // namespace apml
