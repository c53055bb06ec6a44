// Layout of the pieces of the per-sample Sinkhorn kernels, and the device
// routines that place owners and write pairs into it (k_place and
// k_pack_pairs in sinkhorn.hip).
//
// Each row's (column's) pairs are cut into pieces of kSinkPiece consecutive
// pairs; an owner with n pieces takes a group of 2^ceil(log2 n) consecutive
// positions, groups ordered by size (largest first) so that every group is
// aligned to its size. Position p belongs to lane p % kSinkLanes, slot
// p / kSinkLanes. Arrays are plane-major: word w of position p of sample b
// sits at ((b * slots + p / kSinkLanes) * words + w) * kSinkLanes + p % kSinkLanes.
#pragma once

#include "apml_internal.h"

namespace apml {
namespace pieces {

constexpr int kT = kSinkLanes;
constexpr int kP = kSinkPiece;

__device__ __forceinline__ size_t pk_index(int b, int p, int w, int words, int slots)
{
    return (((size_t)b * slots + p / kT) * words + w) * kT + p % kT;
}

// The reverse kernel keeps the adjoint of every pair in LDS at the place of
// the pair in the row pieces: slot s, pair e, lane l at (s * kP + e) * kT + l,
// so that the row phase reads and writes consecutive words; a spare entry
// after them takes the reads and writes of the column pieces' padding.
__host__ __device__ constexpr int adj_slots(int slots) { return slots * kP * kT; }
__device__ __forceinline__ int adj_slot(int p, int e) { return ((p / kT) * kP + e) * kT + p % kT; }

// Placement of the pieces of one order of sample b by one workgroup of kT
// threads: every owner gets the first position of its group (first |
// log2(group) << 16 in place[(b * 2 + order) * kSinkOwners + owner]), the
// info word of every position is written (owner | log2 group << 11 | head <<
// 14 | valid << 15 | first row-major position of a row piece << 16), and the
// P0 / index / position words are cleared (the pack routines fill in the real
// pairs; column padding points at the reverse kernel's spare adjoint). The
// host has checked that the positions fit (slots * kT) and that no owner has
// more than kSinkMaxGroup pieces. hist and base: 8 ints of LDS each.
__device__ inline void place_order(const DevPlan &d, int32_t *place, int b, bool rows, int *hist, int *base)
{
    constexpr int kSL = kSinkOwners / kT; // owners per thread
    const int tid = threadIdx.x;
    const int n_own = rows ? d.N : d.M;
    const int32_t *ptr = rows ? d.row_ptr + (size_t)b * d.N : d.col_ptr + (size_t)b * d.M;
    const PackedOrder pk = rows ? d.pk_row : d.pk_col;
    const int slots = pk.slots, cap = slots * kT;
    const int lo = d.row_ptr[(size_t)b * d.N];
    {
        const size_t np0 = (size_t)slots * kP * kT, ngi = np0 / 2;
        const uint32_t dummy = (uint32_t)adj_slots(slots);
        for (size_t k = tid; k < np0; k += kT)
            pk.p0[(size_t)b * np0 + k] = 0.0f;
        for (size_t k = tid; k < ngi; k += kT) {
            pk.gi[(size_t)b * ngi + k] = 0u;
            if (!rows)
                pk.pos[(size_t)b * ngi + k] = dummy | dummy << 16;
        }
    }
    if (tid < 8)
        hist[tid] = 0;
    __syncthreads();
    int lg[kSL], rk[kSL], st[kSL], len[kSL];
#pragma unroll
    for (int s = 0; s < kSL; ++s) {
        const int k = kSL * tid + s;
        lg[s] = -1;
        if (k < n_own) {
            st[s] = ptr[k];
            len[s] = ptr[k + 1] - st[s];
            lg[s] = sink_log2_group(sink_pieces(len[s]));
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
    for (int s = 0; s < kSL; ++s) {
        if (lg[s] < 0)
            continue;
        const int k = kSL * tid + s, c = 1 << lg[s];
        const int first = base[lg[s]] + (rk[s] << lg[s]);
        place[((size_t)b * 2 + (rows ? 0 : 1)) * kSinkOwners + k] = first | (lg[s] << 16);
        for (int q = 0; q < c; ++q) {
            uint32_t info = (uint32_t)k | ((uint32_t)lg[s] << 11) | ((q == 0 ? 1u : 0u) << 14) | 0x8000u;
            if (rows && q * kP < len[s])
                info |= ((uint32_t)(st[s] + q * kP - lo) & 0xFFFFu) << 16;
            pk.info[pk_index(b, first + q, 0, 1, slots)] = info;
        }
    }
}

// Pair `off` of row i (sample b), with column j and P0, into its row piece.
__device__ __forceinline__ void pack_row_pair(const DevPlan &d, const int32_t *place, int b, int i, int off, int j,
                                              float p0)
{
    const PackedOrder &pk = d.pk_row;
    const int p = (place[((size_t)b * 2) * kSinkOwners + i] & 0xFFFF) + off / kP, e = off % kP;
    pk.p0[pk_index(b, p, e, kP, pk.slots)] = p0;
    uint16_t *gi = reinterpret_cast<uint16_t *>(pk.gi + pk_index(b, p, e / 2, kP / 2, pk.slots));
    gi[e & 1] = (uint16_t)(j << 3); // byte offset of an 8-byte entry
}

// Entry `off` of column j (sample b), with row i, the pair's offset roff in
// its row and P0, into its column piece; its position word is where the
// reverse kernel keeps the pair's adjoint (its row piece).
__device__ __forceinline__ void pack_col_pair(const DevPlan &d, const int32_t *place, int b, int j, int off, int i,
                                              int roff, float p0)
{
    const PackedOrder &pk = d.pk_col;
    const int p = (place[((size_t)b * 2 + 1) * kSinkOwners + j] & 0xFFFF) + off / kP, e = off % kP;
    pk.p0[pk_index(b, p, e, kP, pk.slots)] = p0;
    uint16_t *gi = reinterpret_cast<uint16_t *>(pk.gi + pk_index(b, p, e / 2, kP / 2, pk.slots));
    gi[e & 1] = (uint16_t)(i << 3);
    const int rp = (place[((size_t)b * 2) * kSinkOwners + i] & 0xFFFF) + roff / kP;
    uint16_t *ps = reinterpret_cast<uint16_t *>(pk.pos + pk_index(b, p, e / 2, kP / 2, pk.slots));
    ps[e & 1] = (uint16_t)adj_slot(rp, roff % kP);
}

} // namespace pieces
} // namespace apml
