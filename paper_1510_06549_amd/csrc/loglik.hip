// loglik.hip -- joint log p(W, Z, R) of the current state, fp64 (gfx950).
//
// The collapsed joint of the thesis's blocked-Gibbs derivation with P = I,
// as four sums (each written as fixed-order block partials, then reduced in a
// fixed order, so the value is bit-reproducible):
//   cells     sum_{g,k,w: n>0} log S^n_{t,a} - log C(n, t)
//   base      sum_k lgamma(V gamma) - lgamma(V gamma + B_k)
//                   + sum_w lgamma(gamma + B_wk) - lgamma(gamma)
//   PYP       sum_{g,k} log (b|a)_{T_gk} - log (b)_{N_gk}
//   documents sum_d lgamma(K alpha) - lgamma(K alpha + L_d)
//                   + sum_k lgamma(alpha + n_dk) - lgamma(alpha)
// With word associations (non-identity P^g) the base counts B_wk are keyed by
// each head's source word, and the joint gains the association factor of the
// thesis's joint with the v variables: one p_{g,w,v} per table head,
//   heads     sum_{i: r_i = 1} log p_{g(i), w_i, v_i}.
// A cell with t > n or t = 0 < n (zero probability) sets err[0].
#include "spdp_internal.hpp"

namespace spdp {

namespace {

constexpr int kLBlock = 256;
constexpr int kCellBlocks = 2048;
constexpr int kBaseBlocks = 512;
constexpr int kPypBlocks = 64;
constexpr int kDocBlocks = 2048;  // one document per wave and iteration
constexpr int kHeadBlocks = 1024; // word associations only

__device__ double block_sum(double v)
{
    __shared__ double part[kLBlock / 64];
    for (int o = 32; o > 0; o >>= 1) v += __shfl_down(v, o);
    const int w = threadIdx.x >> 6;
    __syncthreads();
    if ((threadIdx.x & 63) == 0) part[w] = v;
    __syncthreads();
    double s = 0.0;
    if (threadIdx.x == 0)
        for (int i = 0; i < (int)(blockDim.x >> 6); ++i) s += part[i];
    return s;
}

__global__ void __launch_bounds__(kLBlock) k_ll_cells(int64_t ncell, int32_t ncap,
                                                      const int32_t *__restrict__ nt,
                                                      const double *__restrict__ logS,
                                                      const double *__restrict__ lfact,
                                                      double *__restrict__ partial,
                                                      int32_t *__restrict__ err)
{
    double acc = 0.0;
    bool bad = false;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < ncell; i += stride) {
        const int32_t x = nt[i];
        const int32_t nn = x & kCountMax, tt = x >> kCountBits;
        if (nn == 0 && tt == 0) continue;
        if (tt <= 0 || tt > nn || nn > ncap) {
            bad = true;
            continue;
        }
        acc += logS[tri_index(nn, tt)] - (lfact[nn] - lfact[tt] - lfact[nn - tt]);
    }
    if (bad) atomicOr(err, 1);
    const double s = block_sum(acc);
    if (threadIdx.x == 0) partial[blockIdx.x] = s;
}

__global__ void __launch_bounds__(kLBlock) k_ll_base(int32_t V, int32_t K, int32_t Kp,
                                                     double gamma, const int32_t *__restrict__ B,
                                                     const int32_t *__restrict__ Bk,
                                                     double *__restrict__ partial)
{
    double acc = 0.0;
    const double lg0 = lgamma(gamma);
    const int64_t ncell = (int64_t)V * Kp;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < ncell; i += stride) {
        const int32_t x = B[i];
        if (x > 0) acc += lgamma(gamma + (double)x) - lg0;
    }
    if (blockIdx.x == 0) {
        const double Vg = (double)V * gamma;
        for (int32_t k = threadIdx.x; k < K; k += blockDim.x)
            acc += lgamma(Vg) - lgamma(Vg + (double)Bk[k]);
    }
    const double s = block_sum(acc);
    if (threadIdx.x == 0) partial[blockIdx.x] = s;
}

// log (x|y)_T = sum_{j<T} log(x + j y)
__device__ __forceinline__ double log_poch(double x, double y, int32_t T)
{
    if (T <= 0) return 0.0;
    if (y == 0.0) return (double)T * log(x);
    return (double)T * log(y) + lgamma(x / y + (double)T) - lgamma(x / y);
}

__global__ void __launch_bounds__(kLBlock) k_ll_pyp(int32_t G, int32_t K, int32_t Kp, double a,
                                                    double b, const int32_t *__restrict__ Ngk,
                                                    const int32_t *__restrict__ Tgk,
                                                    double *__restrict__ partial)
{
    double acc = 0.0;
    const int64_t nres = (int64_t)G * K;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j < nres; j += stride) {
        const int64_t g = j / K, k = j % K;
        const int64_t idx = g * Kp + k;
        acc += log_poch(b, a, Tgk[idx]) - log_poch(b, 1.0, Ngk[idx]);
    }
    const double s = block_sum(acc);
    if (threadIdx.x == 0) partial[blockIdx.x] = s;
}

// One wave per document (LDS histogram of its topics); documents strided
// over the grid.
__global__ void __launch_bounds__(kLBlock) k_ll_docs(int32_t D, int32_t K, double alpha,
                                                     const int64_t *__restrict__ doc_off,
                                                     const int32_t *__restrict__ zr,
                                                     double *__restrict__ partial)
{
    __shared__ int32_t hist_all[kLBlock / 64][SPDP_MAX_K];
    const int32_t wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int32_t waves = blockDim.x >> 6;
    int32_t *hist = hist_all[wave];
    const double lga = lgamma(alpha), lgKa = lgamma((double)K * alpha);
    double acc = 0.0;
    for (int32_t d = blockIdx.x * waves + wave; d < D; d += gridDim.x * waves) {
        const int64_t beg = doc_off[d], end = doc_off[d + 1];
        for (int32_t k = lane; k < K; k += 64) hist[k] = 0;
        __threadfence_block();
        __builtin_amdgcn_wave_barrier();
        for (int64_t i = beg + lane; i < end; i += 64) atomicAdd(&hist[zr_topic(zr[i])], 1);
        __threadfence_block();
        __builtin_amdgcn_wave_barrier();
        for (int32_t k = lane; k < K; k += 64) {
            const int32_t c = hist[k];
            if (c > 0) acc += lgamma(alpha + (double)c) - lga;
        }
        if (lane == 0) acc += lgKa - lgamma((double)K * alpha + (double)(end - beg));
        __threadfence_block();
        __builtin_amdgcn_wave_barrier();
    }
    const double s = block_sum(acc);
    if (threadIdx.x == 0) partial[blockIdx.x] = s;
}

// sum over table heads of log p of the head's source (word associations)
__global__ void __launch_bounds__(kLBlock) k_ll_heads(int64_t N, int32_t Sp,
                                                      const int32_t *__restrict__ gw,
                                                      const int32_t *__restrict__ zr,
                                                      const double *__restrict__ p64,
                                                      double *__restrict__ partial)
{
    double acc = 0.0;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < N; i += stride) {
        const int32_t v = zr[i];
        if (v & 1) acc += log(p64[(int64_t)gw[i] * Sp + zr_slot(v)]);
    }
    const double s = block_sum(acc);
    if (threadIdx.x == 0) partial[blockIdx.x] = s;
}

__global__ void __launch_bounds__(kLBlock) k_ll_final(int64_t n, const double *__restrict__ partial,
                                                      double *__restrict__ out)
{
    double acc = 0.0;
    for (int64_t i = threadIdx.x; i < n; i += blockDim.x) acc += partial[i];
    const double s = block_sum(acc);
    if (threadIdx.x == 0) *out = s;
}

}  // namespace

int64_t loglik_partials_needed()
{
    return kCellBlocks + kBaseBlocks + kPypBlocks + kDocBlocks + kHeadBlocks;
}

hipError_t launch_loglik(const Model &m, const DeviceBuffers &b, const int32_t *zr,
                         hipStream_t st)
{
    double *p = b.partial;
    hipLaunchKernelGGL(k_ll_cells, dim3(kCellBlocks), dim3(kLBlock), 0, st,
                       (int64_t)m.G * m.V * m.Kp, m.ncap, b.nt, b.logS, b.lfact, p, b.err);
    p += kCellBlocks;
    hipLaunchKernelGGL(k_ll_base, dim3(kBaseBlocks), dim3(kLBlock), 0, st, m.V, m.K, m.Kp, m.gamma,
                       b.B, b.Bk, p);
    p += kBaseBlocks;
    hipLaunchKernelGGL(k_ll_pyp, dim3(kPypBlocks), dim3(kLBlock), 0, st, m.G, m.K, m.Kp, m.a, m.b,
                       b.Ngk, b.Tgk, p);
    p += kPypBlocks;
    hipLaunchKernelGGL(k_ll_docs, dim3(kDocBlocks), dim3(kLBlock), 0, st, m.D, m.K, m.alpha,
                       b.doc_off, zr, p);
    p += kDocBlocks;
    int64_t np = p - b.partial;
    if (m.Sp > 0) {
        hipLaunchKernelGGL(k_ll_heads, dim3(kHeadBlocks), dim3(kLBlock), 0, st, m.N, m.Sp, b.gw,
                           zr, b.p64, p);
        np += kHeadBlocks;
    }
    hipLaunchKernelGGL(k_ll_final, dim3(1), dim3(kLBlock), 0, st, np, b.partial, b.scalar);
    return hipGetLastError();
}

}  // namespace spdp
