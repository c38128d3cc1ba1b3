// sampler_common.hpp -- device helpers shared by the sampling kernels
// (gfx950, wave64): coalesced loads of a lane's slice of a count row, lane
// reads, the DPP wave scan and the interleaved LDS row layout.
#pragma once

#include "spdp_internal.hpp"

namespace spdp {

// Ratio pairs addressable with 32-bit byte offsets (a 4 GiB table): the
// samplers use 64-bit addresses only for a table past this.
constexpr int64_t kSmallQ = 1ll << 29;

// KPL consecutive int32 of one row, loaded with the widest aligned vector
// loads; chunks that start at or beyond the row length are zero.
template <int KPL>
__device__ __forceinline__ void load_slice(int32_t (&v)[KPL], const int32_t *__restrict__ row,
                                           int32_t kbase, int32_t Kp)
{
    if constexpr (KPL % 4 == 0) {
#pragma unroll
        for (int c = 0; c < KPL / 4; ++c) {
            int4 x = make_int4(0, 0, 0, 0);
            if (kbase + 4 * c < Kp) x = *reinterpret_cast<const int4 *>(row + kbase + 4 * c);
            v[4 * c + 0] = x.x;
            v[4 * c + 1] = x.y;
            v[4 * c + 2] = x.z;
            v[4 * c + 3] = x.w;
        }
    } else if constexpr (KPL == 2) {
        int2 x = make_int2(0, 0);
        if (kbase < Kp) x = *reinterpret_cast<const int2 *>(row + kbase);
        v[0] = x.x;
        v[1] = x.y;
    } else {
        static_assert(KPL == 1, "KPL must be 1, 2 or a multiple of 4");
        v[0] = (kbase < Kp) ? row[kbase] : 0;
    }
}

// This lane's KPL cells of a count or shadow-base row for the token loop.
// Every lane issues every load, so the number of loads in flight is the same
// on every path and a wait for one load never has to assume that later ones
// were skipped.  A chunk past the row end reads the row's first chunk instead:
// those cells belong to padding topics, whose weights are zero through the
// zero constants f0 = f1 = 0 whatever the cell values, and the values are
// used as loaded (no select that would wait for the load).
template <int KPL>
__device__ __forceinline__ void load_row(int32_t (&v)[KPL], const int32_t *__restrict__ row,
                                         int32_t kbase, int32_t Kp)
{
    if constexpr (KPL % 4 == 0) {
#pragma unroll
        for (int c = 0; c < KPL / 4; ++c) {
            const int32_t off = (kbase + 4 * c < Kp) ? kbase + 4 * c : 0;
            const int4 x = *reinterpret_cast<const int4 *>(row + off);
            v[4 * c + 0] = x.x;
            v[4 * c + 1] = x.y;
            v[4 * c + 2] = x.z;
            v[4 * c + 3] = x.w;
        }
    } else if constexpr (KPL == 2) {
        const int2 x = *reinterpret_cast<const int2 *>(row + (kbase < Kp ? kbase : 0));
        v[0] = x.x;
        v[1] = x.y;
    } else {
        static_assert(KPL == 1, "KPL must be 1, 2 or a multiple of 4");
        v[0] = row[kbase < Kp ? kbase : 0];
    }
}

// The same for a row of 16-bit counts: this lane's KPL values, two per
// 32-bit word (low half first), with the same unconditional loads.
template <int KPL>
__device__ __forceinline__ void load_half_row(uint32_t (&v)[(KPL + 1) / 2],
                                              const uint16_t *__restrict__ row, int32_t kbase,
                                              int32_t Kp)
{
    constexpr int NW = KPL / 2;
    if constexpr (KPL == 1) {
        v[0] = row[kbase < Kp ? kbase : 0];
    } else if constexpr (NW % 4 == 0) {
#pragma unroll
        for (int c = 0; c < NW / 4; ++c) {
            const int32_t off = (kbase + 8 * c < Kp) ? kbase + 8 * c : 0;
            const uint4 x = *reinterpret_cast<const uint4 *>(row + off);
            v[4 * c + 0] = x.x;
            v[4 * c + 1] = x.y;
            v[4 * c + 2] = x.z;
            v[4 * c + 3] = x.w;
        }
    } else if constexpr (NW % 2 == 0) {
#pragma unroll
        for (int c = 0; c < NW / 2; ++c) {
            const int32_t off = (kbase + 4 * c < Kp) ? kbase + 4 * c : 0;
            const uint2 x = *reinterpret_cast<const uint2 *>(row + off);
            v[2 * c + 0] = x.x;
            v[2 * c + 1] = x.y;
        }
    } else {
        static_assert(KPL == 2, "KPL must be 1, 2 or a multiple of 4");
        v[0] = *reinterpret_cast<const uint32_t *>(row + (kbase < Kp ? kbase : 0));
    }
}

// Start, relative to the lane's first topic, of the cells that chunk c of a
// narrow row read brings (16-bit cells, 16-byte chunks hold eight of them;
// chunks are loaded with the same instructions as a full row's, so a narrow
// row repeats its first chunk of each pair, and with KPL = 12 the third
// chunk holds cells 4 .. 11).
template <int KPL>
__device__ __forceinline__ constexpr int narrow_chunk_start(int c)
{
    return KPL == 12 ? (c == 2 ? 4 : 0) : 8 * (c / 2);
}

// This lane's cells of the count row of (group, word) q for the token loop:
// the 32-bit cells (load_row), or, if `narrow` (wave-uniform), the 16-bit
// copy, read with the same load instructions into the same registers so that
// the loads in flight are the same on both paths; the copy's cells, two per
// 32-bit word, are turned into 32-bit cells by widen_cells once they arrive.
// A narrow read can run up to 8 cells past the lane's slice (into the next
// lane's cells, the next row, or the 16-bit buffer's tail padding); chunks
// that start past the row end read the row's first chunk, as in load_row.
template <int KPL>
__device__ __forceinline__ void load_count_row(int32_t (&v)[KPL], const int32_t *__restrict__ nt,
                                               const uint16_t *__restrict__ nt16, int64_t q,
                                               int32_t kbase, int32_t Kp, bool narrow)
{
    const char *row = narrow ? reinterpret_cast<const char *>(nt16 + q * Kp)
                             : reinterpret_cast<const char *>(nt + q * Kp);
    if constexpr (KPL % 4 == 0) {
#pragma unroll
        for (int c = 0; c < KPL / 4; ++c) {
            const int32_t cw = kbase + 4 * c, cn = kbase + narrow_chunk_start<KPL>(c);
            const int32_t off = narrow ? 2 * (cn < Kp ? cn : 0) : 4 * (cw < Kp ? cw : 0);
            const int4 x = *reinterpret_cast<const int4 *>(row + off);
            v[4 * c + 0] = x.x;
            v[4 * c + 1] = x.y;
            v[4 * c + 2] = x.z;
            v[4 * c + 3] = x.w;
        }
    } else if constexpr (KPL == 2) {
        const int32_t k = kbase < Kp ? kbase : 0;
        const int2 x = *reinterpret_cast<const int2 *>(row + (narrow ? 2 * k : 4 * k));
        v[0] = x.x;
        v[1] = x.y;
    } else {
        static_assert(KPL == 1, "KPL must be 1, 2 or a multiple of 4");
        const int32_t k = kbase < Kp ? kbase : 0;
        v[0] = *reinterpret_cast<const int32_t *>(row + (narrow ? 2 * (k & ~1) : 4 * k));
    }
}

// The cells of a narrow row read by load_count_row as packed n | t << 16
// cells (KPL = 1 reads the aligned pair holding its cell).
template <int KPL>
__device__ __forceinline__ void widen_cells(int32_t (&v)[KPL], int32_t kbase)
{
    uint32_t w[KPL];
#pragma unroll
    for (int j = 0; j < KPL; ++j) w[j] = (uint32_t)v[j];
#pragma unroll
    for (int j = 0; j < KPL; ++j) {
        int src;
        if constexpr (KPL % 8 == 0) src = 8 * (j / 8) + (j % 8) / 2;
        else if constexpr (KPL == 12) src = j < 8 ? j / 2 : 10 + (j - 8) / 2;
        else src = j / 2;
        const bool hi = (KPL == 1) ? (kbase & 1) != 0 : (j & 1) != 0;
        v[j] = wide_of(hi ? (w[src] >> 16) : (w[src] & 0xFFFFu));
    }
}

template <int KPL>
__device__ __forceinline__ void load_slice_f(float (&s)[KPL], const float *__restrict__ row,
                                             int32_t kbase, int32_t Kp)
{
    int32_t tmp[KPL];
    load_slice<KPL>(tmp, reinterpret_cast<const int32_t *>(row), kbase, Kp);
#pragma unroll
    for (int j = 0; j < KPL; ++j) s[j] = __int_as_float(tmp[j]);
}

// Element j of a register array for a j that is not a compile-time constant:
// a chain of selects, since indexing the array would place it in scratch
// memory (the empty asm keeps each element an opaque register value, so that
// the compiler does not turn the chain back into an indexed access).
template <typename T, int N>
__device__ __forceinline__ T pick(const T (&v)[N], int j)
{
    T r = v[0];
    asm volatile("" : "+v"(r));
#pragma unroll
    for (int i = 1; i < N; ++i) {
        T x = v[i];
        asm volatile("" : "+v"(x));
        r = (j == i) ? x : r;
    }
    return r;
}

// Index of the fp64 ratio pair of a cell with nn customers and tt tables
// (the token removed); an empty cell takes pair (0, 0) = (0, 1).
__device__ __forceinline__ int64_t exact_q_index(const ExactCtx &X, int32_t nn, int32_t tt)
{
    const int32_t n_ = nn <= 0 ? 0 : (nn < X.ncap ? nn : X.ncap - 1);
    const int32_t t_ = tt < 0 ? 0 : (tt > n_ ? n_ : tt);
    return tri_index(n_, t_);
}

__device__ __forceinline__ int32_t readlane(int32_t x, int32_t lane)
{
    return __builtin_amdgcn_readlane(x, lane);
}

__device__ __forceinline__ float readlane_f(float x, int32_t lane)
{
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), lane));
}

// Wave64 inclusive prefix sum with DPP: Hillis-Steele inside each row of 16
// lanes (row_shr 1, 2, 4, 8), then row 0's total into row 1 and row 2's into
// row 3 (row_bcast:15), then lane 31's running total into rows 2 and 3
// (row_bcast:31).  Lanes whose DPP source is disabled add 0.
template <int CTRL, int ROW_MASK, bool BOUND>
__device__ __forceinline__ float dpp_src(float x)
{
    return __int_as_float(
        __builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, ROW_MASK, 0xF, BOUND));
}

__device__ __forceinline__ float wave_inclusive_sum(float x)
{
    x += dpp_src<0x111, 0xF, true>(x);   // row_shr:1
    x += dpp_src<0x112, 0xF, true>(x);   // row_shr:2
    x += dpp_src<0x114, 0xF, true>(x);   // row_shr:4
    x += dpp_src<0x118, 0xF, true>(x);   // row_shr:8
    x += dpp_src<0x142, 0xA, false>(x);  // row_bcast:15 -> rows 1, 3
    x += dpp_src<0x143, 0xC, false>(x);  // row_bcast:31 -> rows 2, 3
    return x;
}

// value of lane - 1 (0 in lane 0)
__device__ __forceinline__ float wave_shift_right(float x) { return dpp_src<0x138, 0xF, true>(x); }

// Interleaved LDS rows: the KPL values of lane l sit in 16-byte chunks
// (chunk c of lane l at (c * 64 + l) * 4), so a wave's vector read of one
// chunk touches 64 consecutive 16-byte words and no bank twice.
template <int KPL>
__device__ __forceinline__ int32_t lds_pos(int32_t k)
{
    const int32_t l = k / KPL, j = k % KPL;
    if constexpr (KPL % 4 == 0) return ((j >> 2) * 64 + l) * 4 + (j & 3);
    else return j * 64 + l;
}

template <int KPL>
__device__ __forceinline__ void lds_row(float (&v)[KPL], const float *base, int32_t lane)
{
    if constexpr (KPL % 4 == 0) {
#pragma unroll
        for (int c = 0; c < KPL / 4; ++c) {
            const float4 x = reinterpret_cast<const float4 *>(base)[c * 64 + lane];
            v[4 * c + 0] = x.x;
            v[4 * c + 1] = x.y;
            v[4 * c + 2] = x.z;
            v[4 * c + 3] = x.w;
        }
    } else {
#pragma unroll
        for (int j = 0; j < KPL; ++j) v[j] = base[j * 64 + lane];
    }
}

}  // namespace spdp
