// setup.hip -- state construction and count maintenance kernels (gfx950).
//
//   make_gw        token -> count-row index g V + w, per-(g, w) token counts
//   stirling       log S^n_{t,a} rows (fp64 recurrence of the PYP joint,
//                  Corollary 17 passage) and the folded ratio pairs used by the
//                  sampler (Eq. SPDP-sampling-w-z-r0 / -r1 with P = I)
//   init_z         initial topics from Philox (purpose INIT), r = 0
//   totals         N_gk, T_gk by an LDS-privatised histogram; B_k = sum_g T_gk
//   factors        per-(g, k) sweep constants of the conditionals
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

// ----------------------------------------------------------------- fills
template <typename T>
__global__ void k_fill(T *__restrict__ p, int64_t n, T v)
{
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) p[i] = v;
}

template <typename T>
hipError_t fill(T *p, int64_t n, T v, hipStream_t st)
{
    if (n <= 0) return hipSuccess;
    int64_t nb = blocks_for(n, kBlock);
    if (nb > 65536) nb = 65536;
    hipLaunchKernelGGL(k_fill<T>, dim3((unsigned)nb), dim3(kBlock), 0, st, p, n, v);
    return hipGetLastError();
}

// ---------------------------------------------------------------- make_gw
// One block per document: row index per token, validation, per-row counts.
__global__ void k_make_gw(int32_t D, int32_t V, int32_t G, const int32_t *__restrict__ words,
                          const int64_t *__restrict__ doc_off, const int32_t *__restrict__ doc_group,
                          int32_t *__restrict__ gw, int32_t *__restrict__ gw_count,
                          int32_t *__restrict__ bad)
{
    const int32_t d = blockIdx.x;
    if (d >= D) return;
    const int32_t g = doc_group[d];
    const int64_t beg = doc_off[d], end = doc_off[d + 1];
    if (g < 0 || g >= G) {
        if (threadIdx.x == 0) atomicOr(bad, 1);
        return;
    }
    for (int64_t i = beg + threadIdx.x; i < end; i += blockDim.x) {
        const int32_t w = words[i];
        if (w < 0 || w >= V) {
            atomicOr(bad, 2);
            gw[i] = 0;
            continue;
        }
        const int32_t q = g * V + w;
        gw[i] = q;
        atomicAdd(gw_count + q, 1);
    }
}

// ------------------------------------------------------------ narrow rows
// A row is narrow if its (group, word) pair occurs at most kNarrowMax times:
// no count of the row can then exceed kNarrowMax.
__global__ void k_row_narrow(int64_t rows, const int32_t *__restrict__ gw_count,
                             uint8_t *__restrict__ row_narrow, unsigned long long *__restrict__ n)
{
    const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const bool nar = q < rows && gw_count[q] <= kNarrowMax;
    if (q < rows) row_narrow[q] = nar ? 1 : 0;
    const unsigned long long c = __popcll(__ballot(nar));
    if ((threadIdx.x & 63) == 0 && c) atomicAdd(n, c);
}

__global__ void k_tok_narrow(int64_t N, const int32_t *__restrict__ gw,
                             const uint8_t *__restrict__ row_narrow,
                             uint8_t *__restrict__ tok_narrow)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < N) tok_narrow[i] = row_narrow[gw[i]];
}

// --------------------------------------------------------------- max int32
__global__ void k_max_i32(const int32_t *__restrict__ x, int64_t n, int32_t *__restrict__ out)
{
    int32_t m = 0;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride)
        m = max(m, x[i]);
    for (int o = 32; o > 0; o >>= 1) m = max(m, __shfl_xor(m, o));
    if ((threadIdx.x & 63) == 0) atomicMax(out, m);
}

// --------------------------------------------------------------- Stirling
// One workgroup walks the rows: row n + 1 from row n,
//   S^{n+1}_t = S^n_{t-1} + (n - t a) S^n_t,  S^n_0 = [n == 0],  S^n_t = 0 (t > n),
// in log space (log-sum-exp of the two terms).
__global__ void __launch_bounds__(1024) k_stirling_rows(int32_t nmax, double a,
                                                        double *__restrict__ logS)
{
    if (threadIdx.x == 0) logS[0] = 0.0;
    __syncthreads();
    for (int64_t n = 0; n < nmax; ++n) {
        const double *row = logS + tri_index(n, 0);
        double *next = logS + tri_index(n + 1, 0);
        for (int64_t t = threadIdx.x; t <= n + 1; t += blockDim.x) {
            double v;
            if (t == 0) {
                v = -INFINITY;
            } else {
                const double left = row[t - 1];
                const double same = (t <= n) ? row[t] : -INFINITY;
                const double term = (same == -INFINITY) ? -INFINITY
                                                        : same + log((double)n - (double)t * a);
                if (left == -INFINITY) v = term;
                else if (term == -INFINITY) v = left;
                else {
                    const double hi = fmax(left, term), lo = fmin(left, term);
                    v = hi + log1p(exp(lo - hi));
                }
            }
            next[t] = v;
        }
        __threadfence_block();
        __syncthreads();
    }
}

// Folded ratio pairs for 0 <= t <= n < nmax, computed in fp64:
//   Q0(n, t) = (n - t + 1)/(n + 1) * S^{n+1}_t / S^n_t        (outcome r = 0)
//   Q1(n, t) = (t + 1)/(n + 1) * S^{n+1}_{t+1} / S^n_t        (outcome r = 1)
// with Q(0, 0) = (0, 1); entries with t = 0 < n (no valid state) are (0, 0).
// Q holds them rounded once to fp32 (the sampling path), Q64 in fp64 (the
// boundary path), each factor evaluated as the conditional states it: the
// count ratio divided out, times the exponential of the log-table difference.
__global__ void k_stirling_pairs(int32_t nmax, const double *__restrict__ logS,
                                 float2 *__restrict__ Q, double2 *__restrict__ Q64)
{
    const int64_t n = blockIdx.y;
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (n >= nmax || t > n) return;
    float2 q;
    double2 q64;
    if (n == 0) {
        q = make_float2(0.0f, 1.0f);
        q64 = make_double2(0.0, 1.0);
    } else if (t == 0) {
        q = make_float2(0.0f, 0.0f);
        q64 = make_double2(0.0, 0.0);
    } else {
        const double base = logS[tri_index(n, t)];
        const double r0 = exp(logS[tri_index(n + 1, t)] - base);
        const double r1 = exp(logS[tri_index(n + 1, t + 1)] - base);
        const double inv = 1.0 / (double)(n + 1);
        q = make_float2((float)((double)(n - t + 1) * inv * r0), (float)((double)(t + 1) * inv * r1));
        q64 = make_double2((double)(n - t + 1) / (double)(n + 1) * r0,
                           (double)(t + 1) / (double)(n + 1) * r1);
    }
    Q[tri_index(n, t)] = q;
    Q64[tri_index(n, t)] = q64;
}

__global__ void k_lfact(int32_t nmax, double *__restrict__ lfact)
{
    const int64_t n = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (n <= nmax) lfact[n] = lgamma((double)n + 1.0);
}

// ----------------------------------------------------------------- init z
__global__ void k_init_z(int64_t N, int32_t K, uint64_t seed, int32_t *__restrict__ zr)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= N) return;
    const uint32_t x = philox_x0(seed, (uint64_t)i, 0u, kPurposeInit);
    const int32_t z = (int32_t)(((uint64_t)x * (uint64_t)K) >> 32);
    zr[i] = zr_pack(z, 0);
}

__global__ void k_pack_zr(int64_t N, int32_t K, const int32_t *__restrict__ z,
                          const uint8_t *__restrict__ r, int32_t *__restrict__ zr,
                          int32_t *__restrict__ bad)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= N) return;
    int32_t zi = z[i];
    int32_t ri = r[i];
    if (zi < 0 || zi >= K || ri > 1) {
        atomicOr(bad, 4);
        zi = 0;
        ri = 0;
    }
    zr[i] = zr_pack(zi, ri);
}

// Word associations: (z, r, s) -> zr; a head's slot must hold a source of its
// row (p > 0), a token with r = 0 stores slot 0.
__global__ void k_pack_zrs(int64_t N, int32_t K, int32_t Sp, const int32_t *__restrict__ gw,
                           const double *__restrict__ p64, const int32_t *__restrict__ z,
                           const uint8_t *__restrict__ r, const uint8_t *__restrict__ s,
                           int32_t *__restrict__ zr, int32_t *__restrict__ bad)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= N) return;
    int32_t zi = z[i];
    int32_t ri = r[i];
    int32_t si = s ? (int32_t)s[i] : 0;
    if (ri == 0) si = 0;
    if (zi < 0 || zi >= K || ri > 1 || si >= Sp || !(p64[(int64_t)gw[i] * Sp + si] > 0.0)) {
        atomicOr(bad, 4);
        zi = 0;
        ri = 0;
        si = 0;
    }
    zr[i] = zr_pack(zi, ri, si);
}

__global__ void k_unpack_slot(int64_t N, const int32_t *__restrict__ zr, uint8_t *__restrict__ s)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= N) return;
    s[i] = (uint8_t)zr_slot(zr[i]);
}

__global__ void k_unpack_zr(int64_t N, const int32_t *__restrict__ zr, int32_t *__restrict__ z,
                            uint8_t *__restrict__ r)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= N) return;
    const int32_t v = zr[i];
    if (z) z[i] = zr_topic(v);
    if (r) r[i] = (uint8_t)(v & 1);
}

// ----------------------------------------------------------------- totals
// Per block, a chunk of at most 65535 tokens is histogrammed into LDS bins of
// (g, k), each bin packing customers (low 16 bits) and tables (high 16 bits);
// non-zero bins are flushed with global atomics.
constexpr int kTotalsChunk = 32768;

__global__ void __launch_bounds__(1024) k_totals_lds(int64_t N, int32_t Kp, int32_t bins,
                                                     FastDiv divV, const int32_t *__restrict__ gw,
                                                     const int32_t *__restrict__ zr,
                                                     int32_t *__restrict__ Ngk,
                                                     int32_t *__restrict__ Tgk)
{
    extern __shared__ uint32_t h[];
    for (int j = threadIdx.x; j < bins; j += blockDim.x) h[j] = 0u;
    __syncthreads();
    const int64_t beg = (int64_t)blockIdx.x * kTotalsChunk;
    const int64_t end = min(beg + (int64_t)kTotalsChunk, N);
    for (int64_t i = beg + threadIdx.x; i < end; i += blockDim.x) {
        const int32_t v = zr[i];
        const int32_t g = (int32_t)fastdiv((uint32_t)gw[i], divV);
        atomicAdd(&h[g * Kp + zr_topic(v)], 1u + ((uint32_t)(v & 1) << 16));
    }
    __syncthreads();
    for (int j = threadIdx.x; j < bins; j += blockDim.x) {
        const uint32_t x = h[j];
        if (x) {
            atomicAdd(Ngk + j, (int32_t)(x & 0xFFFFu));
            if (x >> 16) atomicAdd(Tgk + j, (int32_t)(x >> 16));
        }
    }
}

__global__ void k_totals_global(int64_t N, int32_t Kp, FastDiv divV,
                                const int32_t *__restrict__ gw, const int32_t *__restrict__ zr,
                                int32_t *__restrict__ Ngk, int32_t *__restrict__ Tgk)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= N) return;
    const int32_t v = zr[i];
    const int32_t g = (int32_t)fastdiv((uint32_t)gw[i], divV);
    atomicAdd(Ngk + g * Kp + zr_topic(v), 1);
    if (v & 1) atomicAdd(Tgk + g * Kp + zr_topic(v), 1);
}

__global__ void k_topic_tables(int32_t G, int32_t Kp, const int32_t *__restrict__ Tgk,
                               int32_t *__restrict__ Bk)
{
    const int32_t k = blockIdx.x * blockDim.x + threadIdx.x;
    if (k >= Kp) return;
    int32_t s = 0;
    for (int32_t g = 0; g < G; ++g) s += Tgk[(int64_t)g * Kp + k];
    Bk[k] = s;
}

// ---------------------------------------------------------------- factors
// Per-(g, k) constants of the conditionals, computed in fp64 and rounded once:
//   f0 = 1 / (b + N_gk),   f1 = (b + a T_gk) / (b + N_gk) / (V gamma + B_k)
// and, for the topic a token is removed from (N >= 1 there),
//   fk[0] = 1 / (b + N - 1)
//   fk[1] = (b + a T) / (b + N - 1) / (V gamma + B_k)            (r = 0 removed)
//   fk[2] = (b + a (T - 1)) / (b + N - 1) / (V gamma + B_k - 1)  (r = 1 removed)
// Padding topics (k >= K) get 0, so their outcomes carry zero weight.
__global__ void k_factors(int32_t G, int32_t K, int32_t Kp, double a, double b, double Vgamma,
                          const int32_t *__restrict__ Ngk, const int32_t *__restrict__ Tgk,
                          const int32_t *__restrict__ Bk, float *__restrict__ f0,
                          float *__restrict__ f1, float *__restrict__ fk)
{
    const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t GK = (int64_t)G * Kp;
    if (j >= GK) return;
    const int32_t k = (int32_t)(j % Kp);
    if (k >= K) {
        f0[j] = f1[j] = 0.0f;
        fk[j] = fk[GK + j] = fk[2 * GK + j] = 0.0f;
        return;
    }
    const double N = (double)Ngk[j], T = (double)Tgk[j], B = (double)Bk[k];
    const double inv = 1.0 / (b + N);
    f0[j] = (float)inv;
    f1[j] = (float)((b + a * T) * inv / (Vgamma + B));
    if (Ngk[j] >= 1) {
        const double invm = 1.0 / (b + N - 1.0);
        fk[j] = (float)invm;
        fk[GK + j] = (float)((b + a * T) * invm / (Vgamma + B));
        fk[2 * GK + j] =
            Tgk[j] >= 1 ? (float)((b + a * (T - 1.0)) * invm / (Vgamma + B - 1.0)) : 0.0f;
    } else {
        fk[j] = fk[GK + j] = fk[2 * GK + j] = 0.0f;
    }
}

}  // namespace

// ======================================================================
// launchers
// ======================================================================
hipError_t launch_fill_i32(int32_t *p, int64_t n, int32_t v, hipStream_t st) { return fill(p, n, v, st); }
hipError_t launch_fill_u32(uint32_t *p, int64_t n, uint32_t v, hipStream_t st) { return fill(p, n, v, st); }
hipError_t launch_fill_u64(unsigned long long *p, int64_t n, unsigned long long v, hipStream_t st)
{
    return fill(p, n, v, st);
}

hipError_t launch_make_gw(const Model &m, const int32_t *words, const int64_t *doc_off,
                          const int32_t *doc_group, int32_t *gw, int32_t *gw_count, int32_t *bad,
                          hipStream_t st)
{
    if (m.D <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_make_gw, dim3(m.D), dim3(kBlock), 0, st, m.D, m.V, m.G, words, doc_off,
                       doc_group, gw, gw_count, bad);
    return hipGetLastError();
}

hipError_t launch_max_i32(const int32_t *x, int64_t n, int32_t *out, hipStream_t st)
{
    int64_t nb = blocks_for(n, kBlock);
    if (nb > 4096) nb = 4096;
    hipLaunchKernelGGL(k_max_i32, dim3((unsigned)nb), dim3(kBlock), 0, st, x, n, out);
    return hipGetLastError();
}

hipError_t launch_stirling(const Model &m, double *logS, float2 *Q, double2 *Q64, double *lfact,
                           hipStream_t st)
{
    const int32_t nmax = m.ncap;  // rows 0..ncap of log S; pairs for n < ncap
    hipLaunchKernelGGL(k_stirling_rows, dim3(1), dim3(1024), 0, st, nmax, m.a, logS);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    dim3 grid((unsigned)blocks_for(nmax, kBlock), (unsigned)nmax);
    hipLaunchKernelGGL(k_stirling_pairs, grid, dim3(kBlock), 0, st, nmax, logS, Q, Q64);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_lfact, dim3((unsigned)blocks_for(nmax + 1, kBlock)), dim3(kBlock), 0, st,
                       nmax, lfact);
    return hipGetLastError();
}

hipError_t launch_init_z(const Model &m, uint64_t seed, int32_t *zr, hipStream_t st)
{
    if (m.N <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_init_z, dim3((unsigned)blocks_for(m.N, kBlock)), dim3(kBlock), 0, st, m.N,
                       m.K, seed, zr);
    return hipGetLastError();
}

hipError_t launch_pack_zr(const Model &m, const int32_t *z, const uint8_t *r, int32_t *zr,
                          int32_t *bad, hipStream_t st)
{
    if (m.N <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_pack_zr, dim3((unsigned)blocks_for(m.N, kBlock)), dim3(kBlock), 0, st, m.N,
                       m.K, z, r, zr, bad);
    return hipGetLastError();
}

hipError_t launch_pack_zrs(const Model &m, const DeviceBuffers &b, const int32_t *z,
                           const uint8_t *r, const uint8_t *s, int32_t *zr, int32_t *bad,
                           hipStream_t st)
{
    if (m.N <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_pack_zrs, dim3((unsigned)blocks_for(m.N, kBlock)), dim3(kBlock), 0, st,
                       m.N, m.K, m.Sp, b.gw, b.p64, z, r, s, zr, bad);
    return hipGetLastError();
}

hipError_t launch_unpack_slot(const Model &m, const int32_t *zr, uint8_t *s, hipStream_t st)
{
    if (m.N <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_unpack_slot, dim3((unsigned)blocks_for(m.N, kBlock)), dim3(kBlock), 0, st,
                       m.N, zr, s);
    return hipGetLastError();
}

hipError_t launch_unpack_zr(const Model &m, const int32_t *zr, int32_t *z, uint8_t *r,
                            hipStream_t st)
{
    if (m.N <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_unpack_zr, dim3((unsigned)blocks_for(m.N, kBlock)), dim3(kBlock), 0, st,
                       m.N, zr, z, r);
    return hipGetLastError();
}

hipError_t launch_totals(const Model &m, const DeviceBuffers &b, const int32_t *zr, hipStream_t st)
{
    return launch_totals_into(m, b, zr, b.Ngk, b.Tgk, b.Bk, st);
}

hipError_t launch_totals_into(const Model &m, const DeviceBuffers &b, const int32_t *zr,
                              int32_t *Ngk, int32_t *Tgk, int32_t *Bk, hipStream_t st)
{
    hipError_t e;
    const int64_t bins = (int64_t)m.G * m.Kp;
    if ((e = fill(Ngk, bins, 0, st)) != hipSuccess) return e;
    if ((e = fill(Tgk, bins, 0, st)) != hipSuccess) return e;
    if (m.N > 0) {
        // (if the queries fail, lds_max stays 0 and the global-atomic histogram runs)
        int dev = 0, lds_max = 0;
        (void)hipGetDevice(&dev);
        (void)hipDeviceGetAttribute(&lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, dev);
        const int64_t lds = bins * (int64_t)sizeof(uint32_t);
        if (lds <= lds_max && lds <= 96 * 1024) {
            const unsigned nb = (unsigned)blocks_for(m.N, kTotalsChunk);
            hipLaunchKernelGGL(k_totals_lds, dim3(nb), dim3(1024), (size_t)lds, st, m.N, m.Kp,
                               (int32_t)bins, m.divV, b.gw, zr, Ngk, Tgk);
        } else {
            hipLaunchKernelGGL(k_totals_global, dim3((unsigned)blocks_for(m.N, kBlock)), dim3(kBlock),
                               0, st, m.N, m.Kp, m.divV, b.gw, zr, Ngk, Tgk);
        }
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    hipLaunchKernelGGL(k_topic_tables, dim3((unsigned)blocks_for(m.Kp, kBlock)), dim3(kBlock), 0, st,
                       m.G, m.Kp, Tgk, Bk);
    return hipGetLastError();
}

hipError_t launch_narrow_flags(const Model &m, const int32_t *gw, const int32_t *gw_count,
                               uint8_t *row_narrow, uint8_t *tok_narrow,
                               unsigned long long *n_narrow, hipStream_t st)
{
    const int64_t rows = (int64_t)m.G * m.V;
    hipLaunchKernelGGL(k_row_narrow, dim3((unsigned)blocks_for(rows, kBlock)), dim3(kBlock), 0, st,
                       rows, gw_count, row_narrow, n_narrow);
    if (m.N > 0)
        hipLaunchKernelGGL(k_tok_narrow, dim3((unsigned)blocks_for(m.N, kBlock)), dim3(kBlock), 0,
                           st, m.N, gw, row_narrow, tok_narrow);
    return hipGetLastError();
}

hipError_t launch_factors(const Model &m, const DeviceBuffers &b, hipStream_t st)
{
    const int64_t n = (int64_t)m.G * m.Kp;
    hipLaunchKernelGGL(k_factors, dim3((unsigned)blocks_for(n, kBlock)), dim3(kBlock), 0, st, m.G,
                       m.K, m.Kp, m.a, m.b, (double)m.V * m.gamma, b.Ngk, b.Tgk, b.Bk, b.f0, b.f1,
                       b.fk);
    return hipGetLastError();
}

}  // namespace spdp
