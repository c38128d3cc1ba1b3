// counts.hip -- exact count maintenance (gfx950).
//
// The customer and table counts of the thesis's collapsed joint are pure
// functions of the per-token state (z, r).  They are held packed, one int32
// per cell: n in the low 16 bits, t in the high 16 bits (every count is
// bounded by the largest per-(group, word) token count, checked < 2^16 at
// creation).
//
//   row index   tokens grouped by count row q = g V + w (row offsets by an
//               exclusive scan of the per-row token counts, then a scatter
//               with one atomic cursor per row; the order inside a row is
//               free, since nothing below depends on it), built once
//   k_route     the sampled states copied into row buckets (see below), so
//               that the rebuild's per-token gathers stay within a region of
//               the cache's size (the plain model)
//   k_rows      per row: LDS histogram of its tokens' (z, r) -> the row's
//               packed cells; then every cell left with customers but no table
//               promotes the smallest-index token of that cell to table head
//               (the repair of the parallel pass); the row is written (a
//               narrow row only as its 16-bit copy, which the samplers read;
//               its 32-bit row is rewritten from it by k_widen when an entry
//               point reads it), and its table counts are added to the shadow
//               base B[w][k] = sum_g t[g][w][k] (integer atomics, zeroed
//               before, so the sum does not depend on their order)
//   k_rows_assoc
//               the same with word associations: shadow-base counts keyed by
//               each head's source word, and a promoted head takes its row's
//               most probable source
//   k_base16    the 16-bit copy of B the samplers read, min(B, 65535), with a
//               flag raised when a count does not fit (the samplers then read
//               B itself, the plain one only where the copy saturates)
//   k_unpack    export of n and t as separate int32 arrays, [k][w] per group
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

// The row's tokens' states, four per lane in flight: lane l takes row list
// entries rs + l, rs + l + 64, ... and hands each (token index, state v) to f
// in any order.  The states are read from their routed copy zr_b, where the
// states of the rows of one bucket sit together (row_slot: the copy's slot of
// each row list entry).
template <typename F>
__device__ __forceinline__ void for_row_states(int32_t rs, int32_t re, int32_t lane,
                                               const int32_t *__restrict__ perm,
                                               const int32_t *__restrict__ row_slot,
                                               const uint16_t *__restrict__ zr_b, F &&f)
{
    int32_t j = rs + lane;
    for (; j + 192 < re; j += 256) {
        int32_t t[4], s[4], v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            t[u] = perm[j + 64 * u];
            s[u] = row_slot[j + 64 * u];
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) v[u] = (int32_t)zr_b[s[u]];
#pragma unroll
        for (int u = 0; u < 4; ++u) f(t[u], v[u]);
    }
    for (; j < re; j += 64) f(perm[j], (int32_t)zr_b[row_slot[j]]);
}

// The same, gathering each state from token order (the word-association
// rebuild, whose time is set by its atomics into B rather than by these
// gathers, so that routing the states first does not pay there).
template <typename F>
__device__ __forceinline__ void for_row_states_direct(int32_t rs, int32_t re, int32_t lane,
                                                      const int32_t *__restrict__ perm,
                                                      const int32_t *__restrict__ zr, F &&f)
{
    int32_t j = rs + lane;
    for (; j + 192 < re; j += 256) {
        int32_t t[4], v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) t[u] = perm[j + 64 * u];
#pragma unroll
        for (int u = 0; u < 4; ++u) v[u] = zr[t[u]];
#pragma unroll
        for (int u = 0; u < 4; ++u) f(t[u], v[u]);
    }
    for (; j < re; j += 64) {
        const int32_t t = perm[j];
        f(t, zr[t]);
    }
}

// ------------------------------------------------------- state route
// The rebuild reads each row's states in row order, while the sampler writes
// them in token order.  Gathering them one 4-byte state at a time from token
// order fetches a whole line per state; instead the plain model's rebuild
// first copies the states (k_route, coalesced reads, writes in runs) into
// zr_b, where the states of each bucket of rows (the rows starting in one
// window of 2^kRouteShift row positions) occupy that bucket's range of row
// positions, so that the rows' gathers stay within a region that fits the
// cache.  Without word associations a state is z << 1 | r < 2^11 (K <= 1024),
// so the copy holds it in 16 bits: a bucket is about 4 MB, and a cache line
// serves 64 states.  The route is static: fixed with the row index.
constexpr int kRouteShift = 21;
static_assert(2 * SPDP_MAX_K - 1 <= 0xFFFF, "a state without a source slot fits in 16 bits");
constexpr int kRouteThreads = 1024;

// start of each bucket's range: the smallest start of its non-empty rows
__global__ void k_bucket_start(int64_t rows, const int32_t *__restrict__ row_off,
                               int32_t *__restrict__ start)
{
    const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (q < rows && row_off[q] < row_off[q + 1])
        atomicMin(&start[row_off[q] >> kRouteShift], row_off[q]);
}

// tok_slot[i]: token i's slot in its bucket's range.  Each block counts its
// tokens per bucket in LDS (nb ints), reserves one run per bucket with a
// global cursor (initialised to the bucket starts), and places its tokens in
// those runs.
__global__ void __launch_bounds__(kRouteThreads) k_route_build(int64_t N, int32_t nb,
                                                               const int32_t *__restrict__ gw,
                                                               const int32_t *__restrict__ row_off,
                                                               int32_t *__restrict__ cursor,
                                                               int32_t *__restrict__ tok_slot)
{
    extern __shared__ int32_t run[];
    for (int32_t k = threadIdx.x; k < nb; k += kRouteThreads) run[k] = 0;
    __syncthreads();
    const int64_t i = (int64_t)blockIdx.x * kRouteThreads + threadIdx.x;
    int32_t bk = 0, local = 0;
    if (i < N) {
        bk = row_off[gw[i]] >> kRouteShift;
        local = atomicAdd(&run[bk], 1);
    }
    __syncthreads();
    for (int32_t k = threadIdx.x; k < nb; k += kRouteThreads) {
        const int32_t c = run[k];
        run[k] = c ? atomicAdd(&cursor[k], c) : 0;
    }
    __syncthreads();
    if (i < N) tok_slot[i] = run[bk] + local;
}

// row_slot[j] = tok_slot[perm[j]]
__global__ void k_compose(int64_t N, const int32_t *__restrict__ perm,
                          const int32_t *__restrict__ tok_slot, int32_t *__restrict__ row_slot)
{
    const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (j < N) row_slot[j] = tok_slot[perm[j]];
}

// zr_b[tok_slot[i]] = zr[i] (as 16 bits), four tokens per thread
__global__ void __launch_bounds__(kBlock) k_route(int64_t N, const int32_t *__restrict__ tok_slot,
                                                  const int32_t *__restrict__ zr,
                                                  uint16_t *__restrict__ zr_b)
{
    const int64_t i0 = (int64_t)blockIdx.x * (4 * kBlock) + threadIdx.x;
    int32_t d[4], v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const int64_t i = i0 + (int64_t)u * kBlock;
        d[u] = i < N ? tok_slot[i] : -1;
        v[u] = i < N ? zr[i] : 0;
    }
#pragma unroll
    for (int u = 0; u < 4; ++u)
        if (d[u] >= 0) zr_b[d[u]] = (uint16_t)v[u];
}

// One 64-lane block per count row; the row's histogram and the smallest token
// index of each topic in LDS (2 Kp ints of dynamic shared memory).  Every
// token's state is read once: a cell left with customers but no table holds
// only r = 0 tokens, and its smallest-index token becomes its head.  Blocks
// are dealt to the 8 XCDs in turn; block b rebuilds row
// (b mod 8) rows_per_xcd + b / 8, so that each XCD walks its own run of rows
// in order and the bucket of routed states its rows gather from stays in that
// XCD's L2 (blocks past the last row return).
__global__ void __launch_bounds__(64) k_rows(int64_t rows, int64_t rows_per_xcd, int32_t V,
                                             int32_t Kp,
                                             const int32_t *__restrict__ row_off,
                                             const int32_t *__restrict__ perm,
                                             const int32_t *__restrict__ row_slot,
                                             const uint16_t *__restrict__ zr_b,
                                             const uint8_t *__restrict__ row_narrow,
                                             int32_t *__restrict__ zr, int32_t *__restrict__ nt,
                                             uint16_t *__restrict__ nt16, int32_t *__restrict__ B,
                                             uint32_t *__restrict__ rep_part)
{
    extern __shared__ int32_t rows_lds[];
    int32_t *h = rows_lds, *first = rows_lds + Kp;
    const int64_t q = (int64_t)(blockIdx.x & 7) * rows_per_xcd + (blockIdx.x >> 3);
    if (q >= rows) return;
    const int32_t lane = threadIdx.x;
    const int32_t rs = row_off[q], re = row_off[q + 1];
    uint32_t rep = 0;
    if (rs < re) {
        for (int32_t k = lane; k < Kp; k += 64) {
            h[k] = 0;
            first[k] = INT_MAX;
        }
        __syncthreads();
        // the gathers at wave priority 2, so that a row's loads leave ahead of
        // the other wavefronts' row writes
        __builtin_amdgcn_s_setprio(2);
        for_row_states(rs, re, lane, perm, row_slot, zr_b, [&](int32_t tok, int32_t v) {
            atomicAdd(&h[v >> 1], 1 + ((v & 1) << 16));
            atomicMin(&first[v >> 1], tok);
        });
        __builtin_amdgcn_s_setprio(0);
        __syncthreads();
        int32_t *__restrict__ row = nt + q * Kp;
        uint16_t *__restrict__ row16 = nt16 + q * Kp;
        int32_t *__restrict__ base = B + (q % V) * Kp;
        const bool nar = row_narrow[q] != 0;
        for (int32_t k = lane; k < Kp; k += 64) {
            int32_t x = h[k];
            if (x != 0 && (x >> 16) == 0) {
                const int32_t tok = first[k];
                zr[tok] = zr[tok] | 1;
                x += 1 << 16;
                ++rep;
            }
            if (nar) row16[k] = narrow_of(x);
            else row[k] = x;
            if (x >> 16) atomicAdd(&base[k], x >> 16);
        }
    }
    for (int o = 32; o > 0; o >>= 1) rep += __shfl_xor(rep, o);
    if (lane == 0) rep_part[q] = rep;
}

// Word associations: the same per-row rebuild, where a promoted head takes
// the row's most probable source (head_slot[q]) and every head adds one to
// the shadow-base count of its source, B[src][k] (zeroed before; integer
// atomics, so the result does not depend on their order).
__global__ void __launch_bounds__(64) k_rows_assoc(int32_t Kp, int32_t Sp,
                                                   const int32_t *__restrict__ row_off,
                                                   const int32_t *__restrict__ perm,
                                                   const int32_t *__restrict__ srcrec,
                                                   const uint8_t *__restrict__ head_slot,
                                                   const uint8_t *__restrict__ row_narrow,
                                                   int32_t *__restrict__ zr,
                                                   int32_t *__restrict__ nt,
                                                   uint16_t *__restrict__ nt16,
                                                   int32_t *__restrict__ B,
                                                   uint32_t *__restrict__ rep_part)
{
    extern __shared__ int32_t rows_lds[];
    int32_t *h = rows_lds, *first = rows_lds + Kp;
    const int64_t q = blockIdx.x;
    const int32_t lane = threadIdx.x;
    const int32_t rs = row_off[q], re = row_off[q + 1];
    const int32_t *__restrict__ src = srcrec + q * 2 * Sp;
    uint32_t rep = 0;
    if (rs < re) {
        for (int32_t k = lane; k < Kp; k += 64) {
            h[k] = 0;
            first[k] = INT_MAX;
        }
        __syncthreads();
        for_row_states_direct(rs, re, lane, perm, zr, [&](int32_t tok, int32_t v) {
            const int32_t k = zr_topic(v);
            atomicAdd(&h[k], 1 + ((v & 1) << 16));
            atomicMin(&first[k], tok);
            if (v & 1) atomicAdd(&B[(int64_t)src[zr_slot(v)] * Kp + k], 1);
        });
        __syncthreads();
        const int32_t hs = head_slot[q];
        int32_t *__restrict__ row = nt + q * Kp;
        uint16_t *__restrict__ row16 = nt16 + q * Kp;
        const bool nar = row_narrow[q] != 0;
        for (int32_t k = lane; k < Kp; k += 64) {
            int32_t x = h[k];
            if (x != 0 && (x >> 16) == 0) {
                const int32_t tok = first[k];
                zr[tok] = zr_pack(k, 1, hs);
                x += 1 << 16;
                atomicAdd(&B[(int64_t)src[hs] * Kp + k], 1);
                ++rep;
            }
            if (nar) row16[k] = narrow_of(x);
            else row[k] = x;
        }
    }
    for (int o = 32; o > 0; o >>= 1) rep += __shfl_xor(rep, o);
    if (lane == 0) rep_part[q] = rep;
}

// B16 = min(B, 65535), *wide = 1 if any B > 65535 (B already built)
__global__ void k_base16(int64_t cells, const int32_t *__restrict__ B,
                         uint16_t *__restrict__ B16, int32_t *__restrict__ wide)
{
    const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    bool over = false;
    if (j < cells) {
        const int32_t s = B[j];
        over = s > 0xFFFF;
        B16[j] = (uint16_t)(over ? 0xFFFF : s);
    }
    if (__any(over) && (threadIdx.x & 63) == 0) atomicOr(wide, 1);
}

// The 32-bit rows of the narrow rows, rewritten from their 16-bit copies (one
// block per row; rows that are not narrow are skipped).
__global__ void k_widen(int32_t Kp, const uint8_t *__restrict__ row_narrow,
                        const uint16_t *__restrict__ nt16, int32_t *__restrict__ nt)
{
    const int64_t q = blockIdx.x;
    if (!row_narrow[q]) return;
    for (int32_t k = threadIdx.x; k < Kp; k += blockDim.x)
        nt[q * Kp + k] = wide_of(nt16[q * Kp + k]);
}

// Export of one group's counts as [k][w] (topic-major, the thesis's logical
// order): a 64 x 64 tile of cells is read along topics (rows are contiguous
// in k) and written along words through LDS, so both sides are coalesced.
__global__ void __launch_bounds__(256) k_unpack(int32_t V, int32_t K, int32_t Kp,
                                                const int32_t *__restrict__ nt_g,
                                                int32_t *__restrict__ n_out,
                                                int32_t *__restrict__ t_out)
{
    __shared__ int32_t tile[64][65];
    const int32_t tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
    const int32_t w0 = blockIdx.x * 64, k0 = blockIdx.y * 64;
    for (int32_t i = ty; i < 64; i += 4) {
        const int32_t w = w0 + i, k = k0 + tx;
        tile[i][tx] = (w < V && k < K) ? nt_g[(int64_t)w * Kp + k] : 0;
    }
    __syncthreads();
    for (int32_t i = ty; i < 64; i += 4) {
        const int32_t k = k0 + i, w = w0 + tx;
        if (k >= K || w >= V) continue;
        const int32_t x = tile[tx][i];
        const int64_t j = (int64_t)k * V + w;
        if (n_out) n_out[j] = x & 0xFFFF;
        if (t_out) t_out[j] = x >> 16;
    }
}

// Sum of x[0..n) into *out (fixed-order two-level reduction).
__global__ void __launch_bounds__(kBlock) k_sum_u32(const uint32_t *__restrict__ x, int64_t n,
                                                    unsigned long long *__restrict__ part)
{
    unsigned long long s = 0;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) s += x[i];
    for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o);
    __shared__ unsigned long long p[kBlock / 64];
    if ((threadIdx.x & 63) == 0) p[threadIdx.x >> 6] = s;
    __syncthreads();
    if (threadIdx.x == 0) {
        unsigned long long t = 0;
        for (int j = 0; j < kBlock / 64; ++j) t += p[j];
        part[blockIdx.x] = t;
    }
}

__global__ void __launch_bounds__(kBlock) k_count_diff(const int32_t *__restrict__ a,
                                                       const int32_t *__restrict__ b, int64_t n,
                                                       unsigned long long *__restrict__ part)
{
    unsigned long long s = 0;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride)
        s += (a[i] != b[i]) ? 1ull : 0ull;
    for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o);
    __shared__ unsigned long long p[kBlock / 64];
    if ((threadIdx.x & 63) == 0) p[threadIdx.x >> 6] = s;
    __syncthreads();
    if (threadIdx.x == 0) {
        unsigned long long t = 0;
        for (int j = 0; j < kBlock / 64; ++j) t += p[j];
        part[blockIdx.x] = t;
    }
}

__global__ void __launch_bounds__(kBlock) k_sum_u64(const unsigned long long *__restrict__ part,
                                                    int n, unsigned long long *__restrict__ out)
{
    __shared__ unsigned long long p[kBlock];
    unsigned long long s = 0;
    for (int i = threadIdx.x; i < n; i += blockDim.x) s += part[i];
    p[threadIdx.x] = s;
    __syncthreads();
    if (threadIdx.x == 0) {
        unsigned long long t = 0;
        for (int j = 0; j < kBlock; ++j) t += p[j];
        *out = t;
    }
}

constexpr int kReduceBlocks = 1024;

// ------------------------------------------------------- exclusive scan
// Three passes over tiles of kScanTile ints: tile sums, a one-block scan of
// the tile sums (in place, exclusive), and the tiles' own scans offset by
// their tile's prefix.  Totals must fit in int32.
constexpr int kScanThreads = 256;
constexpr int kScanItems = 16;
constexpr int kScanTile = kScanThreads * kScanItems;

// Block-wide exclusive scan of one int per thread; the block's total is
// returned to every thread.
__device__ int32_t block_exclusive_scan(int32_t x, int32_t *total)
{
    __shared__ int32_t warp_sums[kScanThreads / 64];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    int32_t incl = x;
    for (int o = 1; o < 64; o <<= 1) {
        const int32_t y = __shfl_up(incl, o);
        if (lane >= o) incl += y;
    }
    __syncthreads();
    if (lane == 63) warp_sums[w] = incl;
    __syncthreads();
    int32_t before = 0, all = 0;
    for (int i = 0; i < kScanThreads / 64; ++i) {
        const int32_t v = warp_sums[i];
        if (i < w) before += v;
        all += v;
    }
    *total = all;
    return before + incl - x;
}

__global__ void __launch_bounds__(kScanThreads) k_tile_sums(const int32_t *__restrict__ in,
                                                            int64_t n, int32_t *__restrict__ sums)
{
    const int64_t t0 = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
    int32_t s = 0;
    for (int i = 0; i < kScanItems; ++i)
        if (t0 + i < n) s += in[t0 + i];
    int32_t total = 0;
    (void)block_exclusive_scan(s, &total);
    if (threadIdx.x == 0) sums[blockIdx.x] = total;
}

__global__ void __launch_bounds__(kScanThreads) k_scan_sums(int32_t *__restrict__ sums, int64_t nb)
{
    int32_t carry = 0;
    for (int64_t b0 = 0; b0 < nb; b0 += kScanThreads) {
        const int64_t j = b0 + threadIdx.x;
        const int32_t x = j < nb ? sums[j] : 0;
        int32_t total = 0;
        const int32_t ex = block_exclusive_scan(x, &total);
        if (j < nb) sums[j] = carry + ex;
        carry += total;
    }
}

__global__ void __launch_bounds__(kScanThreads) k_tile_scan(const int32_t *__restrict__ in,
                                                            int64_t n,
                                                            const int32_t *__restrict__ sums,
                                                            int32_t *__restrict__ out)
{
    const int64_t t0 = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
    int32_t v[kScanItems], s = 0;
    for (int i = 0; i < kScanItems; ++i) {
        v[i] = t0 + i < n ? in[t0 + i] : 0;
        s += v[i];
    }
    int32_t total = 0;
    int32_t run = sums[blockIdx.x] + block_exclusive_scan(s, &total);
    for (int i = 0; i < kScanItems; ++i) {
        if (t0 + i < n) out[t0 + i] = run;
        run += v[i];
    }
}

// token i goes to the next free slot of its row
__global__ void k_scatter_rows(int64_t N, const int32_t *__restrict__ gw,
                               int32_t *__restrict__ cursor, int32_t *__restrict__ perm)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < N) perm[atomicAdd(&cursor[gw[i]], 1)] = (int32_t)i;
}

// ------------------------------------------------------- visiting order
constexpr int kOrderThreads = 1024;
constexpr int kOrderChunk = 4096;  // documents per chunk (4 per thread)
constexpr int kOrderItems = kOrderChunk / kOrderThreads;

// Block-wide exclusive scan for the order kernels (1024 threads).
__device__ int32_t order_exclusive_scan(int32_t x, int32_t *total)
{
    __shared__ int32_t wsum[kOrderThreads / 64];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    int32_t incl = x;
    for (int o = 1; o < 64; o <<= 1) {
        const int32_t y = __shfl_up(incl, o);
        if (lane >= o) incl += y;
    }
    __syncthreads();
    if (lane == 63) wsum[w] = incl;
    __syncthreads();
    int32_t before = 0, all = 0;
    for (int i = 0; i < kOrderThreads / 64; ++i) {
        const int32_t v = wsum[i];
        if (i < w) before += v;
        all += v;
    }
    *total = all;
    return before + incl - x;
}

// lengths of this thread's documents of chunk blockIdx.x (0 past the end)
__device__ __forceinline__ void chunk_lengths(int32_t D, const int64_t *__restrict__ doc_off,
                                              int32_t (&len)[kOrderItems], int32_t &longest)
{
    const int64_t d0 = (int64_t)blockIdx.x * kOrderChunk + (int64_t)threadIdx.x * kOrderItems;
    int32_t mx = 0;
    for (int i = 0; i < kOrderItems; ++i) {
        const int64_t d = d0 + i;
        len[i] = d < D ? (int32_t)(doc_off[d + 1] - doc_off[d]) : 0;
        mx = max(mx, len[i]);
    }
    __shared__ int32_t lmax;
    if (threadIdx.x == 0) lmax = 0;
    __syncthreads();
    atomicMax(&lmax, mx);
    __syncthreads();
    longest = lmax;
}

// cnt[c][p] = documents of chunk c longer than p (p < L)
__global__ void __launch_bounds__(kOrderThreads) k_order_counts(int32_t D, int32_t L,
                                                                const int64_t *__restrict__ doc_off,
                                                                int32_t *__restrict__ cnt)
{
    int32_t len[kOrderItems], longest = 0;
    chunk_lengths(D, doc_off, len, longest);
    int32_t *row = cnt + (int64_t)blockIdx.x * L;
    for (int32_t p = 0; p < L; ++p) {
        if (p >= longest) {  // (uniform: no document of the chunk reaches p)
            for (int32_t q = p + threadIdx.x; q < L; q += kOrderThreads) row[q] = 0;
            break;
        }
        int32_t x = 0;
        for (int i = 0; i < kOrderItems; ++i) x += len[i] > p ? 1 : 0;
        int32_t total = 0;
        (void)order_exclusive_scan(x, &total);
        if (threadIdx.x == 0) row[p] = total;
    }
}

// cnt[c][p] -> first slot of chunk c's documents at position p (position p
// starts after every token of positions < p; chunks in order within it);
// base[p] = that start
__global__ void __launch_bounds__(kOrderThreads) k_order_offsets(int32_t chunks, int32_t L,
                                                                 int32_t *__restrict__ cnt,
                                                                 int32_t *__restrict__ base)
{
    // per position: exclusive scan over chunks (one thread per position)
    for (int32_t p = threadIdx.x; p < L; p += kOrderThreads) {
        int32_t run = 0;
        for (int32_t c = 0; c < chunks; ++c) {
            const int32_t x = cnt[(int64_t)c * L + p];
            cnt[(int64_t)c * L + p] = run;
            run += x;
        }
        base[p] = run;  // tokens at position p
    }
    __syncthreads();
    // positions' starts: exclusive scan of the per-position token counts
    int32_t carry = 0;
    for (int32_t p0 = 0; p0 < L; p0 += kOrderThreads) {
        const int32_t p = p0 + threadIdx.x;
        const int32_t x = p < L ? base[p] : 0;
        int32_t total = 0;
        const int32_t ex = order_exclusive_scan(x, &total);
        __syncthreads();
        if (p < L) base[p] = carry + ex;
        carry += total;
        __syncthreads();
    }
}

__global__ void __launch_bounds__(kOrderThreads) k_order_place(int32_t D, int32_t L,
                                                               const int64_t *__restrict__ doc_off,
                                                               const int32_t *__restrict__ cnt,
                                                               const int32_t *__restrict__ base,
                                                               int32_t *__restrict__ order)
{
    int32_t len[kOrderItems], longest = 0;
    chunk_lengths(D, doc_off, len, longest);
    const int64_t d0 = (int64_t)blockIdx.x * kOrderChunk + (int64_t)threadIdx.x * kOrderItems;
    const int32_t *row = cnt + (int64_t)blockIdx.x * L;
    for (int32_t p = 0; p < longest; ++p) {
        int32_t x = 0;
        for (int i = 0; i < kOrderItems; ++i) x += len[i] > p ? 1 : 0;
        int32_t total = 0;
        int32_t slot = base[p] + row[p] + order_exclusive_scan(x, &total);
        for (int i = 0; i < kOrderItems; ++i)
            if (len[i] > p) order[slot++] = (int32_t)(doc_off[d0 + i] + p);
    }
}

}  // namespace

hipError_t exclusive_scan(const int32_t *in, int32_t *out, int64_t n, hipStream_t st)
{
    if (n <= 0) return hipSuccess;
    const int64_t nb = (n + kScanTile - 1) / kScanTile;
    int32_t *sums = nullptr;
    hipError_t e = hipMalloc(&sums, (size_t)nb * sizeof(int32_t));
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_tile_sums, dim3((unsigned)nb), dim3(kScanThreads), 0, st, in, n, sums);
    hipLaunchKernelGGL(k_scan_sums, dim3(1), dim3(kScanThreads), 0, st, sums, nb);
    hipLaunchKernelGGL(k_tile_scan, dim3((unsigned)nb), dim3(kScanThreads), 0, st, in, n, sums,
                       out);
    e = hipGetLastError();
    hipError_t e2 = hipStreamSynchronize(st);
    (void)hipFree(sums);
    return e != hipSuccess ? e : e2;
}

hipError_t build_row_index(const Model &m, DeviceBuffers &b, const int32_t *gw_count,
                           hipStream_t st)
{
    const int64_t rows = (int64_t)m.G * m.V;
    // row offsets: exclusive sum of the per-row token counts (rows + 1
    // entries, the last count being zero)
    hipError_t e = exclusive_scan(gw_count, b.row_off, rows + 1, st);
    if (e != hipSuccess || m.N <= 0) return e;
    int32_t *cursor = nullptr;
    if ((e = hipMalloc(&cursor, (size_t)rows * sizeof(int32_t))) != hipSuccess) return e;
    e = hipMemcpyAsync(cursor, b.row_off, (size_t)rows * sizeof(int32_t),
                       hipMemcpyDeviceToDevice, st);
    if (e == hipSuccess) {
        hipLaunchKernelGGL(k_scatter_rows, dim3((unsigned)blocks_for(m.N, kBlock)), dim3(kBlock),
                           0, st, m.N, b.gw, cursor, b.perm);
        e = hipGetLastError();
    }
    hipError_t e2 = hipStreamSynchronize(st);
    (void)hipFree(cursor);
    if (e != hipSuccess || e2 != hipSuccess) return e != hipSuccess ? e : e2;
    if (!b.tok_slot) return hipSuccess;  // no route (word associations)

    // the state route (bucket starts are row starts, so every bucket's tokens
    // fill exactly its range of row positions)
    const int32_t nb = (int32_t)((m.N - 1) >> kRouteShift) + 1;
    int32_t *start = nullptr;
    if ((e = hipMalloc(&start, (size_t)nb * sizeof(int32_t))) != hipSuccess) return e;
    e = launch_fill_i32(start, nb, INT_MAX, st);
    if (e == hipSuccess) {
        hipLaunchKernelGGL(k_bucket_start, dim3((unsigned)blocks_for(rows, kBlock)), dim3(kBlock),
                           0, st, rows, b.row_off, start);
        hipLaunchKernelGGL(k_route_build, dim3((unsigned)blocks_for(m.N, kRouteThreads)),
                           dim3(kRouteThreads), (size_t)nb * sizeof(int32_t), st, m.N, nb, b.gw,
                           b.row_off, start, b.tok_slot);
        hipLaunchKernelGGL(k_compose, dim3((unsigned)blocks_for(m.N, kBlock)), dim3(kBlock), 0, st,
                           m.N, b.perm, b.tok_slot, b.row_slot);
        e = hipGetLastError();
    }
    e2 = hipStreamSynchronize(st);
    (void)hipFree(start);
    return e != hipSuccess ? e : e2;
}

// Visiting order of the asynchronous sweep: tokens by their position inside
// the document, documents in index order at each position (the word order
// rearrangement).  Documents are taken in chunks of kOrderChunk; for every
// position p, chunk c counts its documents longer than p, a scan over chunks
// and over positions gives each (chunk, position) its first slot, and the
// chunk's block ranks its documents longer than p by a block-wide scan.
// Fills b.order and b.tok_doc.
hipError_t build_visit_order(const Model &m, DeviceBuffers &b, hipStream_t st)
{
    if (m.N <= 0) return hipSuccess;
    int32_t *pos = nullptr, *mx = nullptr, *cnt = nullptr, *base = nullptr;
    hipError_t e = hipMalloc(&pos, (size_t)m.N * 4);
    if (e == hipSuccess) e = hipMalloc(&mx, 4);
    if (e == hipSuccess) e = launch_tok_doc(m, b.doc_off, b.tok_doc, pos, st);
    // the longest document bounds the positions
    int32_t longest = 0;
    if (e == hipSuccess) e = launch_fill_i32(mx, 1, 0, st);
    if (e == hipSuccess) e = launch_max_i32(pos, m.N, mx, st);
    if (e == hipSuccess) e = hipMemcpyAsync(&longest, mx, 4, hipMemcpyDeviceToHost, st);
    if (e == hipSuccess) e = hipStreamSynchronize(st);
    const int32_t L = longest + 1;  // positions 0 .. longest
    const int64_t chunks = (m.D + kOrderChunk - 1) / kOrderChunk;
    if (e == hipSuccess) e = hipMalloc(&cnt, (size_t)(chunks * L) * sizeof(int32_t));
    if (e == hipSuccess) e = hipMalloc(&base, (size_t)L * sizeof(int32_t));
    if (e == hipSuccess) {
        hipLaunchKernelGGL(k_order_counts, dim3((unsigned)chunks), dim3(kOrderThreads), 0, st,
                           m.D, L, b.doc_off, cnt);
        hipLaunchKernelGGL(k_order_offsets, dim3(1), dim3(kOrderThreads), 0, st, (int32_t)chunks,
                           L, cnt, base);
        hipLaunchKernelGGL(k_order_place, dim3((unsigned)chunks), dim3(kOrderThreads), 0, st,
                           m.D, L, b.doc_off, cnt, base, b.order);
        e = hipGetLastError();
    }
    hipError_t e2 = hipStreamSynchronize(st);
    (void)hipFree(pos);
    (void)hipFree(mx);
    (void)hipFree(cnt);
    (void)hipFree(base);
    return e != hipSuccess ? e : e2;
}

hipError_t launch_rows(const Model &m, const DeviceBuffers &b, int32_t *zr, hipStream_t st)
{
    const int64_t rows = (int64_t)m.G * m.V;
    hipError_t e = launch_fill_i32(b.B, (int64_t)m.V * m.Kp, 0, st);
    if (e != hipSuccess) return e;
    if (m.N > 0)
        hipLaunchKernelGGL(k_route, dim3((unsigned)blocks_for(m.N, 4 * kBlock)), dim3(kBlock), 0, st,
                           m.N, b.tok_slot, zr, b.zr_b);
    const size_t lds = 2 * (size_t)m.Kp * sizeof(int32_t);
    const int64_t rows_per_xcd = (rows + 7) / 8;
    hipLaunchKernelGGL(k_rows, dim3((unsigned)(8 * rows_per_xcd)), dim3(64), lds, st, rows,
                       rows_per_xcd, m.V, m.Kp, b.row_off, b.perm, b.row_slot, b.zr_b,
                       b.row_narrow, zr, b.nt, b.nt16, b.B, b.rep_part);
    return hipGetLastError();
}

hipError_t launch_widen(const Model &m, const DeviceBuffers &b, hipStream_t st)
{
    const int64_t rows = (int64_t)m.G * m.V;
    hipLaunchKernelGGL(k_widen, dim3((unsigned)rows), dim3(m.Kp < 256 ? (unsigned)m.Kp : 256u), 0,
                       st, m.Kp, b.row_narrow, b.nt16, b.nt);
    return hipGetLastError();
}

hipError_t launch_rows_assoc(const Model &m, const DeviceBuffers &b, int32_t *zr, hipStream_t st)
{
    const int64_t rows = (int64_t)m.G * m.V;
    hipError_t e = launch_fill_i32(b.B, (int64_t)m.V * m.Kp, 0, st);
    if (e != hipSuccess) return e;
    const size_t lds = 2 * (size_t)m.Kp * sizeof(int32_t);
    hipLaunchKernelGGL(k_rows_assoc, dim3((unsigned)rows), dim3(64), lds, st, m.Kp, m.Sp,
                       b.row_off, b.perm, b.srcrec, b.head_slot, b.row_narrow, zr, b.nt, b.nt16,
                       b.B, b.rep_part);
    return hipGetLastError();
}

hipError_t launch_base16(const Model &m, const DeviceBuffers &b, hipStream_t st)
{
    const int64_t cells = (int64_t)m.V * m.Kp;
    hipError_t e = launch_fill_i32(b.wide, 1, 0, st);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_base16, dim3((unsigned)blocks_for(cells, kBlock)), dim3(kBlock), 0, st,
                       cells, b.B, b.B16, b.wide);
    return hipGetLastError();
}

hipError_t launch_unpack_counts(const Model &m, const DeviceBuffers &b, int32_t g,
                                int32_t *n_out, int32_t *t_out, hipStream_t st)
{
    const dim3 grid((unsigned)((m.V + 63) / 64), (unsigned)((m.K + 63) / 64));
    hipLaunchKernelGGL(k_unpack, grid, dim3(256), 0, st, m.V, m.K, m.Kp,
                       b.nt + (int64_t)g * m.V * m.Kp, n_out, t_out);
    return hipGetLastError();
}

hipError_t launch_stat_sums(const Model &m, const DeviceBuffers &b, const int32_t *zr_now,
                            const int32_t *zr_before, hipStream_t st)
{
    // ctr[0] = tokens whose state differs, ctr[1] = heads promoted by repair
    const int64_t rows = (int64_t)m.G * m.V;
    hipLaunchKernelGGL(k_count_diff, dim3(kReduceBlocks), dim3(kBlock), 0, st, zr_now, zr_before,
                       m.N, b.part);
    hipLaunchKernelGGL(k_sum_u64, dim3(1), dim3(kBlock), 0, st, b.part, kReduceBlocks, b.ctr);
    hipLaunchKernelGGL(k_sum_u32, dim3(kReduceBlocks), dim3(kBlock), 0, st, b.rep_part, rows,
                       b.part);
    hipLaunchKernelGGL(k_sum_u64, dim3(1), dim3(kBlock), 0, st, b.part, kReduceBlocks, b.ctr + 1);
    return hipGetLastError();
}

int64_t stat_partials_needed() { return kReduceBlocks; }

}  // namespace spdp
