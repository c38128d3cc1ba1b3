// check.hip -- invariant check of the count state (gfx950).
//
// The counts are pure functions of the per-token state (z, r[, source]), and
// a valid state has 0 <= t <= n and t > 0 exactly when n > 0 in every cell
// (a cell with customers but no table, or more tables than customers, has
// joint probability zero).  The thesis corrects drifting counts on the host
// after each parallel iteration (Algorithm MGPU-DP-SPDP Host regenerates
// them); this check is its read-only counterpart: it recounts and compares
// without changing anything.
//
//   k_check_rows   per count row: LDS recount of its tokens' states against
//                  the stored packed cells (of a narrow row, its 16-bit copy,
//                  the one the rebuild writes and the samplers read); invalid
//                  cells; tokens with a topic out of range or (word
//                  associations) a head whose slot names no source
//   k_check_base   plain model: B[w][k] = sum_g t[g][w][k] over the same
//                  copies, B16 = min(B, 65535), and the width flag
//   k_base_heads / k_cmp_base
//                  word associations: B recounted from the heads' sources
//   k_cmp_i32      recomputed totals against the stored ones
#include <climits>

#include "spdp_internal.hpp"

namespace spdp {

namespace {

constexpr int kBlock = 256;

inline int64_t blocks_for(int64_t n, int per_block)
{
    int64_t b = (n + per_block - 1) / per_block;
    return b < 1 ? 1 : b;
}

__device__ __forceinline__ void add_bad(unsigned long long *bad, bool x)
{
    const unsigned long long c = __popcll(__ballot(x));
    if ((threadIdx.x & 63) == 0 && c) atomicAdd(bad, c);
}

// One 64-lane block per count row (Kp ints of dynamic LDS).
template <bool ASSOC>
__global__ void __launch_bounds__(64) k_check_rows(int32_t K, int32_t Kp, int32_t Sp,
                                                   const int32_t *__restrict__ row_off,
                                                   const int32_t *__restrict__ perm,
                                                   const int32_t *__restrict__ zr,
                                                   const int32_t *__restrict__ nt,
                                                   const uint16_t *__restrict__ nt16,
                                                   const uint8_t *__restrict__ row_narrow,
                                                   const double *__restrict__ p64,
                                                   unsigned long long *__restrict__ bad)
{
    extern __shared__ int32_t h[];
    const int64_t q = blockIdx.x;
    const int32_t lane = threadIdx.x;
    const int32_t rs = row_off[q], re = row_off[q + 1];
    for (int32_t k = lane; k < Kp; k += 64) h[k] = 0;
    __syncthreads();
    for (int32_t base = rs; base < re; base += 64) {
        const int32_t j = base + lane;
        bool wrong = false;
        if (j < re) {
            const int32_t v = zr[perm[j]];
            const int32_t k = zr_topic(v), r = v & 1, sl = zr_slot(v);
            if (k >= K) {
                wrong = true;
            } else {
                if constexpr (ASSOC)
                    wrong = r ? (sl >= Sp || !(p64[q * Sp + sl] > 0.0)) : (sl != 0);
                else
                    wrong = sl != 0;
                atomicAdd(&h[k], 1 + (r << kCountBits));
            }
        }
        add_bad(bad, wrong);
    }
    __syncthreads();
    const bool nar = row_narrow[q] != 0;
    for (int32_t k0 = 0; k0 < Kp; k0 += 64) {
        const int32_t k = k0 + lane;
        bool wrong = false;
        if (k < Kp) {
            const int32_t x = nar ? wide_of(nt16[q * Kp + k]) : nt[q * Kp + k];
            const int32_t n = x & kCountMax, t = x >> kCountBits;
            wrong = x != h[k] || t > n || (t == 0) != (n == 0);
        }
        add_bad(bad, wrong);
    }
}

// B[w][k] against sum_g t[g][w][k] of the stored rows, B16 against min(B,
// 65535); over counts the cells with B > 65535.
__global__ void k_check_base(int32_t G, int32_t V, int32_t Kp, const int32_t *__restrict__ nt,
                             const uint16_t *__restrict__ nt16,
                             const uint8_t *__restrict__ row_narrow,
                             const int32_t *__restrict__ B, const uint16_t *__restrict__ B16,
                             unsigned long long *__restrict__ bad,
                             unsigned long long *__restrict__ over)
{
    const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t cells = (int64_t)V * Kp;
    bool wrong = false, big = false;
    if (j < cells) {
        int32_t s = 0;
        const int64_t w = j / Kp;
        for (int32_t g = 0; g < G; ++g) {
            const int64_t c = (int64_t)g * cells + j;
            s += (row_narrow[(int64_t)g * V + w] ? wide_of(nt16[c]) : nt[c]) >> kCountBits;
        }
        const int32_t b = B[j];
        big = b > 0xFFFF;
        wrong = b != s || B16[j] != (uint16_t)(big ? 0xFFFF : b);
    }
    add_bad(bad, wrong);
    add_bad(over, big);
}

// Word associations: the heads' shadow-base counts B'[src][k] from the states.
__global__ void k_base_heads(int64_t N, int32_t Kp, int32_t Sp, const int32_t *__restrict__ gw,
                             const int32_t *__restrict__ srcrec, const int32_t *__restrict__ zr,
                             int32_t *__restrict__ Bre)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= N) return;
    const int32_t v = zr[i];
    const int32_t sl = zr_slot(v);
    if ((v & 1) && sl < Sp) {
        const int32_t src = srcrec[(int64_t)gw[i] * 2 * Sp + sl];
        atomicAdd(&Bre[(int64_t)src * Kp + zr_topic(v)], 1);
    }
}

__global__ void k_cmp_base(int64_t cells, const int32_t *__restrict__ B,
                           const int32_t *__restrict__ Bre, const uint16_t *__restrict__ B16,
                           unsigned long long *__restrict__ bad,
                           unsigned long long *__restrict__ over)
{
    const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    bool wrong = false, big = false;
    if (j < cells) {
        const int32_t b = B[j];
        big = b > 0xFFFF;
        wrong = b != Bre[j] || B16[j] != (uint16_t)(big ? 0xFFFF : b);
    }
    add_bad(bad, wrong);
    add_bad(over, big);
}

__global__ void k_cmp_i32(int64_t n, const int32_t *__restrict__ a, const int32_t *__restrict__ b,
                          unsigned long long *__restrict__ bad)
{
    const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    add_bad(bad, j < n && a[j] != b[j]);
}

// The width flag: 1 exactly when some B exceeds 65535.
__global__ void k_check_wide(const int32_t *__restrict__ wide,
                             const unsigned long long *__restrict__ over,
                             unsigned long long *__restrict__ bad)
{
    if (threadIdx.x == 0 && ((*wide != 0) != (*over != 0))) atomicAdd(bad, 1ull);
}

}  // namespace

// bad[0]: row cells and token states; bad[1]: totals and shadow base;
// bad[2]: cells with B > 65535 (scratch for the width check).  scratch holds
// 2 G Kp + Kp ints, plus V Kp with word associations.
hipError_t launch_check(const Model &m, const DeviceBuffers &b, const int32_t *zr,
                        int32_t *scratch, unsigned long long *bad, hipStream_t st)
{
    const int64_t rows = (int64_t)m.G * m.V;
    const int64_t gk = (int64_t)m.G * m.Kp, vk = (int64_t)m.V * m.Kp;
    const size_t lds = (size_t)m.Kp * sizeof(int32_t);
    if (m.Sp > 0)
        hipLaunchKernelGGL(k_check_rows<true>, dim3((unsigned)rows), dim3(64), lds, st, m.K, m.Kp,
                           m.Sp, b.row_off, b.perm, zr, b.nt, b.nt16, b.row_narrow, b.p64, bad);
    else
        hipLaunchKernelGGL(k_check_rows<false>, dim3((unsigned)rows), dim3(64), lds, st, m.K, m.Kp,
                           1, b.row_off, b.perm, zr, b.nt, b.nt16, b.row_narrow, b.p64, bad);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    int32_t *N = scratch, *T = scratch + gk, *Bk = scratch + 2 * gk;
    if ((e = launch_totals_into(m, b, zr, N, T, Bk, st)) != hipSuccess) return e;
    hipLaunchKernelGGL(k_cmp_i32, dim3((unsigned)blocks_for(gk, kBlock)), dim3(kBlock), 0, st, gk,
                       N, b.Ngk, bad + 1);
    hipLaunchKernelGGL(k_cmp_i32, dim3((unsigned)blocks_for(gk, kBlock)), dim3(kBlock), 0, st, gk,
                       T, b.Tgk, bad + 1);
    hipLaunchKernelGGL(k_cmp_i32, dim3((unsigned)blocks_for(m.Kp, kBlock)), dim3(kBlock), 0, st,
                       (int64_t)m.Kp, Bk, b.Bk, bad + 1);
    if (m.Sp > 0) {
        int32_t *Bre = scratch + 2 * gk + m.Kp;
        if ((e = launch_fill_i32(Bre, vk, 0, st)) != hipSuccess) return e;
        if (m.N > 0)
            hipLaunchKernelGGL(k_base_heads, dim3((unsigned)blocks_for(m.N, kBlock)), dim3(kBlock),
                               0, st, m.N, m.Kp, m.Sp, b.gw, b.srcrec, zr, Bre);
        hipLaunchKernelGGL(k_cmp_base, dim3((unsigned)blocks_for(vk, kBlock)), dim3(kBlock), 0, st,
                           vk, b.B, Bre, b.B16, bad + 1, bad + 2);
    } else {
        hipLaunchKernelGGL(k_check_base, dim3((unsigned)blocks_for(vk, kBlock)), dim3(kBlock), 0,
                           st, m.G, m.V, m.Kp, b.nt, b.nt16, b.row_narrow, b.B, b.B16, bad + 1,
                           bad + 2);
    }
    hipLaunchKernelGGL(k_check_wide, dim3(1), dim3(64), 0, st, b.wide, bad + 2, bad + 1);
    return hipGetLastError();
}

}  // namespace spdp
