// estimate.hip -- point estimates of a state and held-out perplexity (gfx950).
//
// The estimates after convergence (thesis: Eq. spdp-topic-doc-estimate,
// Eq. spdp-word-topic-estimate and Eq. spdp-group-word-topic-estimate, with
// identity transformation matrices, so q = t):
//   theta[d][k]  = (c_dk + alpha) / (L_d + K alpha)
//   phi0[w][k]   = (gamma + B_wk) / (V gamma + B_k)
//   phi[g][w][k] = (n - a t + (b + a T_gk) phi0[w][k]) / (b + N_gk)
// The group estimate weights the base by (b + a T) / (b + N), the weight of a
// new table in the Pitman-Yor seating rule; the printed a T / (b + N) would
// not sum to one over the words.
//
// Held-out perplexity (section "Perplexity"): each test document is folded in
// with phi fixed at the group estimate of the current state.  Its topics start
// uniform (first Philox word with purpose 3 at counter (test token, 0), times
// K, high 32 bits); each fold-in sweep resamples its tokens in order from
//   p(z_n = k | rest) proportional to (c_k without token n + alpha) phi[g][w_n][k]
// with the uniform of purpose 2 at counter (test token, sweep) and the first k
// whose inclusive prefix sum exceeds u * total; then
//   log p(w_d) = sum_n log sum_k phi[g][w_n][k] theta_d[k]
// with theta_d from the final counts.  All in fp64.  One wavefront per test
// document; the estimates are computed from the count rows on the fly.
//
// With word associations (non-identity P^g) phi0 is over source words and the
// base of group g's Pitman-Yor process is P^g phi0_k:
//   phi[g][w][k] = (n - a t + (b + a T_gk) sum_v p_{g,w,v} phi0[v][k]) / (b + N_gk).
#include "sampler_common.hpp"

namespace spdp {

// fp64 wave scans of the fold-in (the sampler's DPP scan, applied to both
// 32-bit halves of each value).
// Both 32-bit halves move with the same DPP control (a disabled source gives
// 0 in both halves, i.e. +0.0).
template <int CTRL, int ROW_MASK, bool BOUND>
__device__ __forceinline__ double dpp_src64(double x)
{
    const int lo = __builtin_amdgcn_update_dpp(0, __double2loint(x), CTRL, ROW_MASK, 0xF, BOUND);
    const int hi = __builtin_amdgcn_update_dpp(0, __double2hiint(x), CTRL, ROW_MASK, 0xF, BOUND);
    return __hiloint2double(hi, lo);
}

__device__ __forceinline__ double wave_inclusive_sum64(double x)
{
    x += dpp_src64<0x111, 0xF, true>(x);
    x += dpp_src64<0x112, 0xF, true>(x);
    x += dpp_src64<0x114, 0xF, true>(x);
    x += dpp_src64<0x118, 0xF, true>(x);
    x += dpp_src64<0x142, 0xA, false>(x);
    x += dpp_src64<0x143, 0xC, false>(x);
    return x;
}

__device__ __forceinline__ double wave_shift_right64(double x)
{
    return dpp_src64<0x138, 0xF, true>(x);
}

__device__ __forceinline__ double readlane64(double x, int32_t l)
{
    return __hiloint2double(__builtin_amdgcn_readlane(__double2hiint(x), l),
                            __builtin_amdgcn_readlane(__double2loint(x), l));
}


namespace {

constexpr int kBlock = 256;
constexpr uint32_t kPurposeFoldin = 2u, kPurposeFoldinInit = 3u;

inline int64_t blocks_for(int64_t n, int per_block)
{
    int64_t b = (n + per_block - 1) / per_block;
    return b < 1 ? 1 : b;
}

// theta of training documents: one 64-lane block per document
__global__ void __launch_bounds__(64) k_theta(int32_t D, int32_t K, double alpha,
                                              const int64_t *__restrict__ doc_off,
                                              const int32_t *__restrict__ zr,
                                              double *__restrict__ theta)
{
    __shared__ int32_t c[SPDP_MAX_K];
    const int32_t d = blockIdx.x;
    if (d >= D) return;
    for (int32_t k = threadIdx.x; k < K; k += 64) c[k] = 0;
    __syncthreads();
    const int64_t beg = doc_off[d], end = doc_off[d + 1];
    for (int64_t i = beg + threadIdx.x; i < end; i += 64) atomicAdd(&c[zr_topic(zr[i])], 1);
    __syncthreads();
    const double inv = 1.0 / ((double)(end - beg) + (double)K * alpha);
    double *row = theta + (int64_t)d * K;
    for (int32_t k = threadIdx.x; k < K; k += 64) row[k] = ((double)c[k] + alpha) * inv;
}

// phi0 as [V][K]
__global__ void k_phi0(int32_t V, int32_t K, int32_t Kp, double gamma, double Vgamma,
                       const int32_t *__restrict__ B, const int32_t *__restrict__ Bk,
                       double *__restrict__ phi0)
{
    const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (j >= (int64_t)V * K) return;
    const int64_t w = j / K, k = j % K;
    phi0[j] = (gamma + (double)B[w * Kp + k]) / (Vgamma + (double)Bk[k]);
}

// phi of group g as [V][K]
__global__ void k_phig(int32_t g, int32_t V, int32_t K, int32_t Kp, double a, double b,
                       double gamma, double Vgamma, const int32_t *__restrict__ nt,
                       const int32_t *__restrict__ B, const int32_t *__restrict__ Ngk,
                       const int32_t *__restrict__ Tgk, const int32_t *__restrict__ Bk,
                       double *__restrict__ phi)
{
    const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (j >= (int64_t)V * K) return;
    const int64_t w = j / K, k = j % K;
    const int32_t x = nt[((int64_t)g * V + w) * Kp + k];
    const double n = (double)(x & kCountMax), t = (double)(x >> kCountBits);
    const double N = (double)Ngk[(int64_t)g * Kp + k], T = (double)Tgk[(int64_t)g * Kp + k];
    const double p0 = (gamma + (double)B[w * Kp + k]) / (Vgamma + (double)Bk[k]);
    phi[j] = (n - a * t + (b + a * T) * p0) / (b + N);
}

// phi of group g as [V][K] with word associations: the base term sums phi0
// over the sources of row (g, w) (padding slots have p = 0)
__global__ void k_phig_assoc(int32_t g, int32_t V, int32_t K, int32_t Kp, int32_t Sp, double a,
                             double b, double gamma, double Vgamma,
                             const int32_t *__restrict__ nt, const int32_t *__restrict__ B,
                             const int32_t *__restrict__ Ngk, const int32_t *__restrict__ Tgk,
                             const int32_t *__restrict__ Bk, const int32_t *__restrict__ srcrec,
                             const double *__restrict__ p64, double *__restrict__ phi)
{
    const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (j >= (int64_t)V * K) return;
    const int64_t w = j / K, k = j % K;
    const int64_t q = (int64_t)g * V + w;
    const int32_t x = nt[q * Kp + k];
    const double n = (double)(x & kCountMax), t = (double)(x >> kCountBits);
    const double N = (double)Ngk[(int64_t)g * Kp + k], T = (double)Tgk[(int64_t)g * Kp + k];
    const double den = Vgamma + (double)Bk[k];
    double base = 0.0;
    for (int32_t s = 0; s < Sp; ++s) {
        const double pv = p64[q * Sp + s];
        if (pv > 0.0) base += pv * ((gamma + (double)B[(int64_t)srcrec[q * 2 * Sp + s] * Kp + k]) / den);
    }
    phi[j] = (n - a * t + (b + a * T) * base) / (b + N);
}

struct FoldArgs {
    const int32_t *gw;        // [Nt] row index g V + w of each test token
    const int64_t *doc_off;   // [Dt + 1]
    const int32_t *doc_group; // [Dt]
    int32_t *z;               // [Nt] fold-in topics
    double *ll_doc;           // [Dt] log p(w_d)
    const int32_t *nt, *B, *Ngk, *Tgk, *Bk;
    const int32_t *srcrec;    // word associations (Sp > 0): source records
    const double *p64;        //   and fp64 p of each row
    uint64_t seed;
    int32_t D, V, K, Kp, n_sweeps, Sp;
    double alpha, a, b, gamma, Vgamma;
};

// sum over the wave's 64 lanes (the last lane's inclusive prefix sum)
__device__ __forceinline__ double wave_sum(double x)
{
    return readlane64(wave_inclusive_sum64(x), 63);
}

// This lane's slices of the rows a test token's group estimate reads, loaded
// whole (padding chunks re-read the row start; their topics weigh nothing):
// the packed count row of q = g V + w and, with P = I (SP = 0), the int32
// shadow-base row of w; with word associations (SP sources per row) the
// shadow-base rows of the row's sources and their p (a padding slot repeats
// the first source with p = 0).
template <int KPL, int SP>
struct FoldRows {
    static constexpr int NB = SP > 0 ? SP : 1;
    int32_t n[KPL];
    int32_t b[NB][KPL];
    double p[NB];
};

template <int KPL, int SP>
__device__ __forceinline__ void load_fold_rows(const FoldArgs &A, int32_t q, int32_t g,
                                               int32_t kbase, FoldRows<KPL, SP> &R)
{
    load_row<KPL>(R.n, A.nt + (int64_t)q * A.Kp, kbase, A.Kp);
    if constexpr (SP == 0) {
        load_row<KPL>(R.b[0], A.B + (int64_t)(q - g * A.V) * A.Kp, kbase, A.Kp);
    } else {
#pragma unroll
        for (int s = 0; s < SP; ++s) {
            const int32_t v = A.srcrec[(int64_t)q * 2 * SP + s];
            R.p[s] = A.p64[(int64_t)q * SP + s];
            load_row<KPL>(R.b[s], A.B + (int64_t)v * A.Kp, kbase, A.Kp);
        }
    }
}

// The group estimate of this lane's topics: (n - a t)/(b + N) plus the base
// weight times (b + a T)/(b + N)/(V gamma + B_k), the base weight being
// gamma + B[w][k], or with word associations the sum over the sources, in
// slot order, of p (gamma + B[v][k]) for p > 0.
template <int KPL, int SP>
__device__ __forceinline__ void phi_from_rows(const FoldArgs &A, const FoldRows<KPL, SP> &R,
                                              int32_t kbase, const double *inv, const double *base,
                                              double (&ph)[KPL])
{
#pragma unroll
    for (int j = 0; j < KPL; ++j) {
        const int32_t k = kbase + j;
        const double n = (double)(R.n[j] & kCountMax), t = (double)(R.n[j] >> kCountBits);
        double bw;
        if constexpr (SP == 0) {
            bw = A.gamma + (double)R.b[0][j];
        } else {
            bw = 0.0;
#pragma unroll
            for (int s = 0; s < SP; ++s)
                if (R.p[s] > 0.0) bw += R.p[s] * (A.gamma + (double)R.b[s][j]);
        }
        ph[j] = (k < A.K) ? (n - A.a * t) * inv[k] + bw * base[k] : 0.0;
    }
}

// The group estimates of tokens 0 .. nc - 1 of a chunk (row indices in the
// lanes of gw_c), in order, handed to f(x, ph).  Where two register sets of
// rows fit, the rows of token x + 1 are requested before token x is
// evaluated; otherwise each token's rows are loaded together, then used.
template <int KPL, int SP, typename F>
__device__ __forceinline__ void for_chunk_phi(const FoldArgs &A, int32_t g, int32_t kbase,
                                              int32_t gw_c, int32_t nc, const double *inv,
                                              const double *base, F &&f)
{
    constexpr int kRows = SP > 0 ? SP + 1 : 2;
    if constexpr (KPL * kRows > 48) {
        for (int32_t x = 0; x < nc; ++x) {
            FoldRows<KPL, SP> r;
            load_fold_rows<KPL, SP>(A, __builtin_amdgcn_readlane(gw_c, x), g, kbase, r);
            double ph[KPL];
            phi_from_rows<KPL, SP>(A, r, kbase, inv, base, ph);
            f(x, ph);
        }
    } else {
        FoldRows<KPL, SP> ra, rb;
        load_fold_rows<KPL, SP>(A, __builtin_amdgcn_readlane(gw_c, 0), g, kbase, ra);
        for (int32_t x = 0; x < nc; x += 2) {
            const int32_t x1 = x + 1 < nc ? x + 1 : x;
            load_fold_rows<KPL, SP>(A, __builtin_amdgcn_readlane(gw_c, x1), g, kbase, rb);
            {
                double ph[KPL];
                phi_from_rows<KPL, SP>(A, ra, kbase, inv, base, ph);
                f(x, ph);
            }
            if (x + 1 < nc) {
                const int32_t x2 = x + 2 < nc ? x + 2 : x + 1;
                load_fold_rows<KPL, SP>(A, __builtin_amdgcn_readlane(gw_c, x2), g, kbase, ra);
                double ph[KPL];
                phi_from_rows<KPL, SP>(A, rb, kbase, inv, base, ph);
                f(x + 1, ph);
            }
        }
    }
}

template <int KPL, int SP>
__global__ void __launch_bounds__(64) k_foldin(FoldArgs A)
{
    // document counts and the group's per-topic factors 1/(b + N) and
    // (b + a T)/(b + N)/(V gamma + B_k) (zero for padding topics)
    __shared__ int32_t c[64 * KPL];
    __shared__ double inv[64 * KPL];
    __shared__ double base[64 * KPL];
    const int32_t d = blockIdx.x;
    if (d >= A.D) return;
    const int32_t lane = threadIdx.x, kbase = lane * KPL;
    const int64_t beg = A.doc_off[d], end = A.doc_off[d + 1];
    const int32_t g = A.doc_group[d];
#pragma unroll
    for (int j = 0; j < KPL; ++j) {
        const int32_t k = kbase + j;
        c[k] = 0;
        inv[k] = base[k] = 0.0;
        if (k < A.K) {
            const double N = (double)A.Ngk[(int64_t)g * A.Kp + k];
            const double T = (double)A.Tgk[(int64_t)g * A.Kp + k];
            inv[k] = 1.0 / (A.b + N);
            base[k] = (A.b + A.a * T) / (A.b + N) / (A.Vgamma + (double)A.Bk[k]);
        }
    }
    __syncthreads();
    // initial topics
    for (int64_t i = beg + lane; i < end; i += 64) {
        const uint32_t x = philox_x0(A.seed, (uint64_t)i, 0u, kPurposeFoldinInit);
        const int32_t z = (int32_t)(((uint64_t)x * (uint64_t)A.K) >> 32);
        A.z[i] = z;
        atomicAdd(&c[z], 1);
    }
    __syncthreads();

    for (int32_t s = 0; s < A.n_sweeps; ++s) {
        // 64 tokens at a time: lane l reads and writes token cb + l, so each
        // lane sees its own earlier writes
        for (int64_t cb = beg; cb < end; cb += 64) {
            const int32_t nc = (int32_t)min((int64_t)64, end - cb);
            const bool mine = lane < nc;
            const int32_t gw_c = mine ? A.gw[cb + lane] : 0;
            int32_t z_c = mine ? A.z[cb + lane] : 0;
            for_chunk_phi<KPL, SP>(A, g, kbase, gw_c, nc, inv, base, [&](int32_t x,
                                                                            const double(&ph)[KPL]) {
                const int64_t i = cb + x;
                const int32_t k0 = __builtin_amdgcn_readlane(z_c, x);
                double pre[KPL];
                double acc = 0.0;
#pragma unroll
                for (int j = 0; j < KPL; ++j) {
                    const int32_t k = kbase + j;
                    const double cw = (double)(c[k] - (k == k0 ? 1 : 0)) + A.alpha;
                    acc += (k < A.K) ? cw * ph[j] : 0.0;
                    pre[j] = acc;
                }
                const double incl = wave_inclusive_sum64(acc);
                const double excl = wave_shift_right64(incl);
                const double total = readlane64(incl, 63);
                const uint32_t xr = philox_x0(A.seed, (uint64_t)i, (uint32_t)s, kPurposeFoldin);
                const double target = (double)(xr >> 8) * (1.0 / 16777216.0) * total;
                const double rel = target - excl;
                int32_t cnt = 0;
#pragma unroll
                for (int j = 0; j < KPL; ++j) cnt += (pre[j] <= rel) ? 1 : 0;
                const unsigned long long cross = __ballot(cnt < KPL && kbase < A.K);
                int32_t k1 = k0;
                if (cross) {
                    const int32_t L = __ffsll((long long)cross) - 1;
                    k1 = L * KPL + __builtin_amdgcn_readlane(cnt, L);
                }
                if (k1 >= A.K) k1 = k0;  // no crossing (rounding at the very top): keep
                if (lane == x) z_c = k1;
                if (lane == 0 && k1 != k0) {
                    c[k0] -= 1;
                    c[k1] += 1;
                }
            });
            if (mine) A.z[cb + lane] = z_c;
        }
    }
    __syncthreads();

    // log p(w_d) with theta_d from the final counts
    const double tden = 1.0 / ((double)(end - beg) + (double)A.K * A.alpha);
    double th[KPL];
#pragma unroll
    for (int j = 0; j < KPL; ++j)
        th[j] = (kbase + j < A.K) ? ((double)c[kbase + j] + A.alpha) * tden : 0.0;
    double ll = 0.0;
    for (int64_t cb = beg; cb < end; cb += 64) {
        const int32_t nc = (int32_t)min((int64_t)64, end - cb);
        const int32_t gw_c = (lane < nc) ? A.gw[cb + lane] : 0;
        for_chunk_phi<KPL, SP>(A, g, kbase, gw_c, nc, inv, base,
                                  [&](int32_t, const double(&ph)[KPL]) {
                                      double p = 0.0;
#pragma unroll
                                      for (int j = 0; j < KPL; ++j) p += ph[j] * th[j];
                                      ll += log(wave_sum(p));
                                  });
    }
    if (lane == 0) A.ll_doc[d] = ll;
}

template <int KPL>
hipError_t launch_fold(const FoldArgs &A, hipStream_t st)
{
    const dim3 grid((unsigned)A.D);
    switch (A.Sp) {
    case 0: hipLaunchKernelGGL((k_foldin<KPL, 0>), grid, dim3(64), 0, st, A); break;
    case 1: hipLaunchKernelGGL((k_foldin<KPL, 1>), grid, dim3(64), 0, st, A); break;
    case 2: hipLaunchKernelGGL((k_foldin<KPL, 2>), grid, dim3(64), 0, st, A); break;
    case 4: hipLaunchKernelGGL((k_foldin<KPL, 4>), grid, dim3(64), 0, st, A); break;
    case 8: hipLaunchKernelGGL((k_foldin<KPL, 8>), grid, dim3(64), 0, st, A); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_theta(const Model &m, const DeviceBuffers &b, const int32_t *zr, double *theta,
                        hipStream_t st)
{
    if (m.D <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_theta, dim3((unsigned)m.D), dim3(64), 0, st, m.D, m.K, m.alpha,
                       b.doc_off, zr, theta);
    return hipGetLastError();
}

hipError_t launch_phi0(const Model &m, const DeviceBuffers &b, double *phi0, hipStream_t st)
{
    const int64_t n = (int64_t)m.V * m.K;
    hipLaunchKernelGGL(k_phi0, dim3((unsigned)blocks_for(n, kBlock)), dim3(kBlock), 0, st, m.V,
                       m.K, m.Kp, m.gamma, (double)m.V * m.gamma, b.B, b.Bk, phi0);
    return hipGetLastError();
}

hipError_t launch_phig(const Model &m, const DeviceBuffers &b, int32_t g, double *phi,
                       hipStream_t st)
{
    const int64_t n = (int64_t)m.V * m.K;
    if (m.Sp > 0)
        hipLaunchKernelGGL(k_phig_assoc, dim3((unsigned)blocks_for(n, kBlock)), dim3(kBlock), 0,
                           st, g, m.V, m.K, m.Kp, m.Sp, m.a, m.b, m.gamma, (double)m.V * m.gamma,
                           b.nt, b.B, b.Ngk, b.Tgk, b.Bk, b.srcrec, b.p64, phi);
    else
        hipLaunchKernelGGL(k_phig, dim3((unsigned)blocks_for(n, kBlock)), dim3(kBlock), 0, st, g,
                           m.V, m.K, m.Kp, m.a, m.b, m.gamma, (double)m.V * m.gamma, b.nt, b.B,
                           b.Ngk, b.Tgk, b.Bk, phi);
    return hipGetLastError();
}

hipError_t launch_foldin(const Model &m, const DeviceBuffers &b, int32_t D_test,
                         const int32_t *gw, const int64_t *doc_off, const int32_t *doc_group,
                         int32_t n_sweeps, uint64_t seed, int32_t *z, double *ll_doc,
                         hipStream_t st)
{
    if (D_test <= 0) return hipSuccess;
    FoldArgs A;
    A.gw = gw;
    A.doc_off = doc_off;
    A.doc_group = doc_group;
    A.z = z;
    A.ll_doc = ll_doc;
    A.nt = b.nt;
    A.B = b.B;
    A.Ngk = b.Ngk;
    A.Tgk = b.Tgk;
    A.Bk = b.Bk;
    A.srcrec = b.srcrec;
    A.p64 = b.p64;
    A.Sp = m.Sp;
    A.seed = seed;
    A.D = D_test;
    A.V = m.V;
    A.K = m.K;
    A.Kp = m.Kp;
    A.n_sweeps = n_sweeps;
    A.alpha = m.alpha;
    A.a = m.a;
    A.b = m.b;
    A.gamma = m.gamma;
    A.Vgamma = (double)m.V * m.gamma;
    switch (sampler_kpl(m.K)) {
    case 1: return launch_fold<1>(A, st);
    case 2: return launch_fold<2>(A, st);
    case 4: return launch_fold<4>(A, st);
    case 8: return launch_fold<8>(A, st);
    case 12: return launch_fold<12>(A, st);
    default: return launch_fold<16>(A, st);
    }
}

}  // namespace spdp
