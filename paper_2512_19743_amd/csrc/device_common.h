// Device helpers shared by the libapml kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <climits>
#include <cstdint>

namespace apml {

constexpr float kInf = __builtin_huge_valf();

// Squared distance in single precision, as d = a - b per coordinate, then
// dx*dx, fma(dy,dy,.), fma(dz,dz,.). The dense scans and the sparse passes
// evaluate exactly this sequence (the library is built without floating-point
// contraction), so their values agree bit for bit; the argmin decisions rest
// on it.
__device__ __forceinline__ float sqdist_f32(float ax, float ay, float az, float bx, float by,
                                            float bz)
{
    const float dx = ax - bx, dy = ay - by, dz = az - bz;
    float s = dx * dx;
    s = __builtin_fmaf(dy, dy, s);
    s = __builtin_fmaf(dz, dz, s);
    return s;
}

// Cost C = ||a - b||_2 (Sec. III-A) in double precision from float coordinates.
__device__ __forceinline__ double dist_f64(const float *a, const float *b)
{
    const double dx = (double)a[0] - (double)b[0];
    const double dy = (double)a[1] - (double)b[1];
    const double dz = (double)a[2] - (double)b[2];
    return sqrt(dx * dx + dy * dy + dz * dz);
}

__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }

// Number of entries of a[s0, s1) below key: four loads in flight at a time
// (a loop of one load per step waits out every load in turn).
__device__ __forceinline__ int count_below(const int32_t *a, int s0, int s1, int key)
{
    int n = 0, q = s0;
    for (; q + 4 <= s1; q += 4) {
        const int v0 = a[q], v1 = a[q + 1], v2 = a[q + 2], v3 = a[q + 3];
        n += (v0 < key) + (v1 < key) + (v2 < key) + (v3 < key);
    }
    for (; q < s1; ++q)
        n += a[q] < key;
    return n;
}

// Read-only data seen through the constant address space: wave-uniform loads
// from it become scalar loads even in kernels that also store to memory.
template <typename T> using const_ptr = const __attribute__((address_space(4))) T *;
typedef float f32x4 __attribute__((ext_vector_type(4)));
template <typename T> __device__ __forceinline__ const_ptr<T> as_const(const T *p)
{
    return (const_ptr<T>)p;
}

// Reductions over aligned groups of G lanes (G divides 64). Butterfly order:
// every lane of a group ends with the same, order-independent bits.
template <int G> __device__ __forceinline__ double group_sum(double v)
{
#pragma unroll
    for (int o = 1; o < G; o <<= 1)
        v += __shfl_xor(v, o);
    return v;
}

template <int G> __device__ __forceinline__ int group_min(int v)
{
#pragma unroll
    for (int o = 1; o < G; o <<= 1)
        v = min(v, __shfl_xor(v, o));
    return v;
}

__device__ __forceinline__ double wave_sum(double v)
{
    for (int o = 32; o > 0; o >>= 1)
        v += __shfl_xor(v, o);
    return v;
}

// Workgroup barrier that orders LDS accesses only: global stores issued
// before it may still be in flight (use __syncthreads when other threads of
// the workgroup read them back).
__device__ __forceinline__ void lds_barrier()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Barrier for a workgroup that shares data through LDS (LDS_ONLY) or also
// through global memory.
template <bool LDS_ONLY> __device__ __forceinline__ void wg_barrier()
{
    if (LDS_ONLY)
        lds_barrier();
    else
        __syncthreads();
}

// Finds, among the pairs of one segment, the first position whose
// single-precision squared distance equals m1 and the first other position
// whose distance equals m2 (the second order statistic): the minimum and the
// second minimum with ties to the smaller index.
template <int G> struct Argmins {
    int f1 = INT_MAX, g1 = INT_MAX, g2 = INT_MAX;
    __device__ void see(int t, float s, float2 m)
    {
        if (s == m.x && f1 == INT_MAX)
            f1 = t;
        if (s == m.y) {
            if (g1 == INT_MAX)
                g1 = t;
            else if (g2 == INT_MAX)
                g2 = t;
        }
    }
    __device__ void resolve(int *q1, int *q2) const
    {
        *q1 = group_min<G>(f1);
        *q2 = group_min<G>(g1 != *q1 ? g1 : g2);
    }
};

// Workgroups are dealt to the 8 XCDs round robin (workgroup i to XCD i % 8),
// and each XCD has its own L2. This maps the hardware index to a logical one
// under which every XCD receives one contiguous range of the grid, so that
// workgroups sharing data (one sample) share an L2.
constexpr int kXcds = 8;
__device__ __forceinline__ int xcd_contiguous(int bid, int grid)
{
    const int q = grid / kXcds, r = grid % kXcds, x = bid % kXcds;
    return x * q + min(x, r) + bid / kXcds;
}

inline unsigned blocks_for(int64_t n, int per_block) { return (unsigned)((n + per_block - 1) / per_block); }

} // namespace apml
