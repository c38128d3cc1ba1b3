// counts.hip -- exact count maintenance (gfx950).
//
// The customer and table counts of the thesis's collapsed joint are pure
// functions of the per-token state (z, r).  They are held packed, one int32
// per cell: n in the low 16 bits, t in the high 16 bits (every count is
// bounded by the largest per-(group, word) token count, checked < 2^16 at
// creation).
//
//   row index   tokens sorted by count row q = g V + w (stable, so each row's
//               token list is in increasing token index), built once
//   k_rows      per row: LDS histogram of its tokens' (z, r) -> the row's
//               packed cells; then every cell left with customers but no
//               table promotes the smallest-index token of that cell to table
//               head (the repair of the parallel pass), and the row is written
//   k_base      shadow-base table counts B[w][k] = sum_g t[g][w][k], and the
//               16-bit copy the sampler reads (with a flag raised when a count
//               does not fit, in which case the sampler reads B itself)
//   k_rows_assoc / k_base16
//               the same with word associations: shadow-base counts keyed by
//               each head's source word, and a promoted head takes its row's
//               most probable source
//   k_unpack    export of n and t as separate int32 arrays
#include <hipcub/hipcub.hpp>

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

__global__ void k_iota(int32_t *__restrict__ x, int64_t n)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) x[i] = (int32_t)i;
}

// The row's tokens' states, four per lane in flight: lane l takes row list
// entries rs + l, rs + l + 64, ... and hands each (list index j, state v) to
// f in any order.
template <typename F>
__device__ __forceinline__ void for_row_states(int32_t rs, int32_t re, int32_t lane,
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
        for (int u = 0; u < 4; ++u) f(j + 64 * u, v[u]);
    }
    for (; j < re; j += 64) f(j, zr[perm[j]]);
}

// One 64-lane block per count row; the row's histogram and the first list
// index of each topic in LDS (2 Kp ints of dynamic shared memory).  Every
// token's state is read once: a cell left with customers but no table holds
// only r = 0 tokens, and its first token in the row list (the smallest token
// index, the list being a stable sort) becomes its head.
__global__ void __launch_bounds__(64) k_rows(int32_t Kp, const int32_t *__restrict__ row_off,
                                             const int32_t *__restrict__ perm,
                                             int32_t *__restrict__ zr, int32_t *__restrict__ nt,
                                             uint32_t *__restrict__ rep_part)
{
    extern __shared__ int32_t rows_lds[];
    int32_t *h = rows_lds, *first = rows_lds + Kp;
    const int64_t q = blockIdx.x;
    const int32_t lane = threadIdx.x;
    const int32_t rs = row_off[q], re = row_off[q + 1];
    uint32_t rep = 0;
    if (rs < re) {
        for (int32_t k = lane; k < Kp; k += 64) {
            h[k] = 0;
            first[k] = INT_MAX;
        }
        __syncthreads();
        for_row_states(rs, re, lane, perm, zr, [&](int32_t j, int32_t v) {
            atomicAdd(&h[v >> 1], 1 + ((v & 1) << 16));
            atomicMin(&first[v >> 1], j);
        });
        __syncthreads();
        int32_t *__restrict__ row = nt + q * Kp;
        for (int32_t k = lane; k < Kp; k += 64) {
            int32_t x = h[k];
            if (x != 0 && (x >> 16) == 0) {
                const int32_t tok = perm[first[k]];
                zr[tok] = zr[tok] | 1;
                x += 1 << 16;
                ++rep;
            }
            row[k] = x;
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
                                                   int32_t *__restrict__ zr,
                                                   int32_t *__restrict__ nt,
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
        for_row_states(rs, re, lane, perm, zr, [&](int32_t j, int32_t v) {
            const int32_t k = zr_topic(v);
            atomicAdd(&h[k], 1 + ((v & 1) << 16));
            atomicMin(&first[k], j);
            if (v & 1) atomicAdd(&B[(int64_t)src[zr_slot(v)] * Kp + k], 1);
        });
        __syncthreads();
        const int32_t hs = head_slot[q];
        int32_t *__restrict__ row = nt + q * Kp;
        for (int32_t k = lane; k < Kp; k += 64) {
            int32_t x = h[k];
            if (x != 0 && (x >> 16) == 0) {
                const int32_t tok = perm[first[k]];
                zr[tok] = zr_pack(k, 1, hs);
                x += 1 << 16;
                atomicAdd(&B[(int64_t)src[hs] * Kp + k], 1);
                ++rep;
            }
            row[k] = x;
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

// B[w][k] = sum_g t[g][w][k];  B16 = min(B, 65535), *wide = 1 if any B > 65535
__global__ void k_base(int32_t G, int32_t V, int32_t Kp, const int32_t *__restrict__ nt,
                       int32_t *__restrict__ B, uint16_t *__restrict__ B16,
                       int32_t *__restrict__ wide)
{
    const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t cells = (int64_t)V * Kp;
    bool over = false;
    if (j < cells) {
        int32_t s = 0;
        for (int32_t g = 0; g < G; ++g) s += nt[(int64_t)g * cells + j] >> 16;
        B[j] = s;
        over = s > 0xFFFF;
        B16[j] = (uint16_t)(over ? 0xFFFF : s);
    }
    if (__any(over) && (threadIdx.x & 63) == 0) atomicOr(wide, 1);
}

__global__ void k_unpack(int32_t V, int32_t K, int32_t Kp, const int32_t *__restrict__ nt_g,
                         int32_t *__restrict__ n_out, int32_t *__restrict__ t_out)
{
    const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (j >= (int64_t)V * K) return;
    const int64_t w = j / K, k = j % K;
    const int32_t x = nt_g[w * Kp + k];
    if (n_out) n_out[j] = x & 0xFFFF;
    if (t_out) t_out[j] = x >> 16;
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

}  // namespace

hipError_t build_row_index(const Model &m, DeviceBuffers &b, const int32_t *gw_count,
                           hipStream_t st)
{
    const int64_t rows = (int64_t)m.G * m.V;
    hipError_t e;
    // row offsets: exclusive sum of the per-row token counts (rows + 1 entries,
    // the last count being zero)
    size_t scan_bytes = 0;
    e = hipcub::DeviceScan::ExclusiveSum(nullptr, scan_bytes, gw_count, b.row_off, rows + 1, st);
    if (e != hipSuccess) return e;
    // stable radix sort of (row, token) pairs
    int end_bit = 1;
    while ((1ll << end_bit) < rows) ++end_bit;
    int32_t *keys_out = nullptr, *vals_in = nullptr;
    size_t sort_bytes = 0;
    e = hipcub::DeviceRadixSort::SortPairs(nullptr, sort_bytes, b.gw, keys_out, vals_in, b.perm,
                                           (int)m.N, 0, end_bit, st);
    if (e != hipSuccess) return e;
    void *temp = nullptr;
    const size_t temp_bytes = scan_bytes > sort_bytes ? scan_bytes : sort_bytes;
    if ((e = hipMalloc(&temp, temp_bytes > 0 ? temp_bytes : 1)) != hipSuccess) return e;
    if ((e = hipMalloc(&keys_out, (size_t)(m.N > 0 ? m.N : 1) * 4)) != hipSuccess) {
        (void)hipFree(temp);
        return e;
    }
    if ((e = hipMalloc(&vals_in, (size_t)(m.N > 0 ? m.N : 1) * 4)) != hipSuccess) {
        (void)hipFree(temp);
        (void)hipFree(keys_out);
        return e;
    }
    size_t tb = temp_bytes;
    e = hipcub::DeviceScan::ExclusiveSum(temp, tb, gw_count, b.row_off, rows + 1, st);
    if (e == hipSuccess && m.N > 0) {
        hipLaunchKernelGGL(k_iota, dim3((unsigned)blocks_for(m.N, kBlock)), dim3(kBlock), 0, st,
                           vals_in, m.N);
        e = hipGetLastError();
        if (e == hipSuccess) {
            tb = temp_bytes;
            e = hipcub::DeviceRadixSort::SortPairs(temp, tb, b.gw, keys_out, vals_in, b.perm,
                                                   (int)m.N, 0, end_bit, st);
        }
    }
    hipError_t e2 = hipStreamSynchronize(st);
    (void)hipFree(temp);
    (void)hipFree(keys_out);
    (void)hipFree(vals_in);
    return e != hipSuccess ? e : e2;
}

// Visiting order of the asynchronous sweep: tokens stably sorted by their
// position inside the document, so at each position the documents come in
// index order (the word order rearrangement).  Fills b.order and b.tok_doc.
hipError_t build_visit_order(const Model &m, DeviceBuffers &b, hipStream_t st)
{
    if (m.N <= 0) return hipSuccess;
    int32_t *pos = nullptr, *keys_out = nullptr, *vals_in = nullptr;
    void *temp = nullptr;
    hipError_t e = hipMalloc(&pos, (size_t)m.N * 4);
    if (e == hipSuccess) e = hipMalloc(&keys_out, (size_t)m.N * 4);
    if (e == hipSuccess) e = hipMalloc(&vals_in, (size_t)m.N * 4);
    if (e == hipSuccess) e = launch_tok_doc(m, b.doc_off, b.tok_doc, pos, st);
    if (e == hipSuccess) {
        hipLaunchKernelGGL(k_iota, dim3((unsigned)blocks_for(m.N, kBlock)), dim3(kBlock), 0, st,
                           vals_in, m.N);
        e = hipGetLastError();
    }
    // the longest document bounds the keys
    int32_t *mx = nullptr;
    int32_t longest = 0;
    if (e == hipSuccess) e = hipMalloc(&mx, 4);
    if (e == hipSuccess) e = launch_fill_i32(mx, 1, 0, st);
    if (e == hipSuccess) e = launch_max_i32(pos, m.N, mx, st);
    if (e == hipSuccess) e = hipMemcpyAsync(&longest, mx, 4, hipMemcpyDeviceToHost, st);
    if (e == hipSuccess) e = hipStreamSynchronize(st);
    int end_bit = 1;
    while ((1ll << end_bit) <= longest) ++end_bit;
    size_t bytes = 0;
    if (e == hipSuccess)
        e = hipcub::DeviceRadixSort::SortPairs(nullptr, bytes, pos, keys_out, vals_in, b.order,
                                               (int)m.N, 0, end_bit, st);
    if (e == hipSuccess) e = hipMalloc(&temp, bytes > 0 ? bytes : 1);
    if (e == hipSuccess)
        e = hipcub::DeviceRadixSort::SortPairs(temp, bytes, pos, keys_out, vals_in, b.order,
                                               (int)m.N, 0, end_bit, st);
    hipError_t e2 = hipStreamSynchronize(st);
    (void)hipFree(pos);
    (void)hipFree(keys_out);
    (void)hipFree(vals_in);
    (void)hipFree(mx);
    (void)hipFree(temp);
    return e != hipSuccess ? e : e2;
}

hipError_t launch_rows(const Model &m, const DeviceBuffers &b, int32_t *zr, hipStream_t st)
{
    const int64_t rows = (int64_t)m.G * m.V;
    const size_t lds = 2 * (size_t)m.Kp * sizeof(int32_t);
    hipLaunchKernelGGL(k_rows, dim3((unsigned)rows), dim3(64), lds, st, m.Kp, b.row_off, b.perm, zr,
                       b.nt, b.rep_part);
    return hipGetLastError();
}

hipError_t launch_base(const Model &m, const DeviceBuffers &b, hipStream_t st)
{
    const int64_t cells = (int64_t)m.V * m.Kp;
    hipError_t e = launch_fill_i32(b.wide, 1, 0, st);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_base, dim3((unsigned)blocks_for(cells, kBlock)), dim3(kBlock), 0, st, m.G,
                       m.V, m.Kp, b.nt, b.B, b.B16, b.wide);
    return hipGetLastError();
}

hipError_t launch_rows_assoc(const Model &m, const DeviceBuffers &b, int32_t *zr, hipStream_t st)
{
    const int64_t rows = (int64_t)m.G * m.V;
    hipError_t e = launch_fill_i32(b.B, (int64_t)m.V * m.Kp, 0, st);
    if (e != hipSuccess) return e;
    const size_t lds = 2 * (size_t)m.Kp * sizeof(int32_t);
    hipLaunchKernelGGL(k_rows_assoc, dim3((unsigned)rows), dim3(64), lds, st, m.Kp, m.Sp,
                       b.row_off, b.perm, b.srcrec, b.head_slot, zr, b.nt, b.B, b.rep_part);
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
    const int64_t cells = (int64_t)m.V * m.K;
    hipLaunchKernelGGL(k_unpack, dim3((unsigned)blocks_for(cells, kBlock)), dim3(kBlock), 0, st,
                       m.V, m.K, m.Kp, b.nt + (int64_t)g * m.V * m.Kp, n_out, t_out);
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
