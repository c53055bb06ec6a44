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
// per-sample offsets
// ---------------------------------------------------------------------------

constexpr int kOffT = 1024;

// Per sample (blockIdx.x) and direction (blockIdx.y: 0 rows, 1 columns): the
// sample-local exclusive scan of the owners' pair counts into row_ptr /
// col_ptr, the sample's total and its piece counts.
__global__ __launch_bounds__(kOffT) void k_sample_scan(const int32_t *cnt, int S, const int32_t *col_cnt, int N,
                                                       int M, int32_t *row_ptr, int32_t *col_ptr, Readback *rb,
                                                       Readback *rb_host)
{
    __shared__ int wsum[kOffT / 64];
    __shared__ int red[2][kOffT / 64];
    const int b = blockIdx.x, rows = blockIdx.y == 0, tid = threadIdx.x, B = gridDim.x;
    const int lane = lane_id(), wave = tid >> 6;
    const int n = rows ? N : M;
    int32_t *out = rows ? row_ptr + (size_t)b * N : col_ptr + (size_t)b * M;
    int carry = 0, pos = 0, mx = 0;
    for (int base = 0; base < n; base += kOffT) {
        const int k = base + tid;
        int len = 0;
        if (k < n) {
            if (rows) {
                const int32_t *rc = cnt + ((size_t)b * N + k) * S;
                int c = 0;
                if (S % 4 == 0) // the row's chunk counts in 16-byte loads, all in flight together
                    for (; c < S; c += 4) {
                        const int4 v = *reinterpret_cast<const int4 *>(rc + c);
                        len += v.x + v.y + v.z + v.w;
                    }
                for (; c < S; ++c)
                    len += rc[c];
            } else {
                len = col_cnt[(size_t)b * M + k];
            }
            const int np = sink_pieces(len);
            pos += 1 << min(sink_log2_group(np), 30);
            mx = max(mx, np);
        }
        int inc = len;
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
        if (k < n)
            out[k] = carry + before + inc - len;
        carry += all;
    }
    for (int off = 32; off > 0; off >>= 1) {
        pos += __shfl_xor(pos, off);
        mx = max(mx, __shfl_xor(mx, off));
    }
    if (lane == 0) {
        red[0][wave] = pos;
        red[1][wave] = mx;
    }
    __syncthreads();
    if (tid == 0) {
        int a = 0, m = 0;
        for (int w = 0; w < kOffT / 64; ++w) {
            a += red[0][w];
            m = max(m, red[1][w]);
        }
        readback_totals(rb)[(rows ? 0 : B) + b] = carry;
        readback_totals(rb_host)[(rows ? 0 : B) + b] = carry;
        int32_t *pc = readback_pieces(rb_host, B) + 4 * b;
        pc[rows ? 0 : 1] = a;
        pc[rows ? 2 : 3] = m;
    }
}

// Adds each sample's base (pairs of the earlier samples) to its local
// offsets, closes row_ptr / col_ptr with the total and fills the read-back
// offsets and counters.
__global__ __launch_bounds__(kOffT) void k_sample_base(const Counters *ctr, int N, int M, int32_t *row_ptr,
                                                       int32_t *col_ptr, const Readback *rb, Readback *rb_host)
{
    __shared__ int base_s;
    const int b = blockIdx.x, rows = blockIdx.y == 0, tid = threadIdx.x, B = gridDim.x;
    const int64_t *tot = readback_totals(const_cast<Readback *>(rb)) + (rows ? 0 : B);
    if (tid == 0) {
        int64_t base = 0;
        for (int k = 0; k < b; ++k)
            base += tot[k];
        base_s = (int)base; // the host rejects totals beyond int32 before using any offset
        if (rows)
            readback_offsets(rb_host, B)[b] = (int)base;
        if (b == B - 1) {
            const int end = (int)(base + tot[b]);
            (rows ? row_ptr[(size_t)B * N] : col_ptr[(size_t)B * M]) = end;
            if (rows)
                readback_offsets(rb_host, B)[B] = end;
        }
    }
    if (b == 0 && rows) // the counters, word by word over the workgroup
        for (int i = tid; i < (int)(sizeof(Counters) / 4); i += kOffT)
            reinterpret_cast<uint32_t *>(&rb_host->ctr)[i] = reinterpret_cast<const uint32_t *>(ctr)[i];
    __syncthreads();
    const int n = rows ? N : M;
    int32_t *out = rows ? row_ptr + (size_t)b * N : col_ptr + (size_t)b * M;
    for (int k = tid; k < n; k += kOffT)
        out[k] += base_s;
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

void launch_offsets(const int32_t *cnt, int S, const int32_t *col_cnt, const Counters *ctr, int B, int N, int M,
                    int32_t *row_ptr, int32_t *col_ptr, Readback *rb, Readback *rb_host, hipStream_t s)
{
    hipLaunchKernelGGL(k_sample_scan, dim3(B, 2), dim3(kOffT), 0, s, cnt, S, col_cnt, N, M, row_ptr, col_ptr, rb,
                       rb_host);
    hipLaunchKernelGGL(k_sample_base, dim3(B, 2), dim3(kOffT), 0, s, ctr, N, M, row_ptr, col_ptr, rb, rb_host);
}

void launch_csc_build(const DevPlan &d, const BuildArgs &a, hipStream_t s)
{
    // d.col_ptr holds the scan of the column counts (launch_col_scan)
    const unsigned g = blocks_for(d.nnz, kBlock);
    hipLaunchKernelGGL(k_csc_fill, dim3(g), dim3(kBlock), 0, s, d, a);
    hipLaunchKernelGGL(k_csc_sort, dim3(g), dim3(kBlock), 0, s, d, a);
}

void launch_csc_sort(const DevPlan &d, const BuildArgs &a, hipStream_t s)
{
    hipLaunchKernelGGL(k_csc_sort, dim3(blocks_for(d.nnz, kBlock)), dim3(kBlock), 0, s, d, a);
}

void launch_count_support(const int32_t *row_ptr, const uint8_t *flags, int B, int N,
                          unsigned long long *out, hipStream_t s)
{
    hipLaunchKernelGGL(k_count_support, dim3(B), dim3(kBlock), 0, s, row_ptr, flags, N, out);
}

} // namespace apml
