// sample_async.hip -- the thesis's asynchronous sweep (an ablation of the
// snapshot sweep), gfx950 wave64.
//
// The scheme of the thesis's parallel word sampling: every token is taken up
// by its own work-group, which reads the global counts as they are at that
// moment, removes its token from them with atomics, computes the 2K
// conditionals (Eq. SPDP-sampling-w-z-r0 / -r1, P = I), draws, and adds the
// token back at its new cell with atomics; no locks, so concurrent tokens read
// each other's partial updates.  Tokens are taken up in the order of the word
// order rearrangement (round robin over the position inside the document), so
// tokens in flight together mostly come from different documents.  The counts
// are regenerated exactly from the new state after the pass (the library's
// row rebuild with its repair), as the thesis's host does after each
// iteration.
//
// Here each wavefront takes the tokens at visiting positions w, w + W, w + 2W,
// ... (W wavefronts in the grid), one at a time.  With W = 1 the pass is
// sequential in the visiting order, because every read of a count happens
// after the previous token's atomics have completed: the atomics return their
// old values and the wave waits for them, and count reads are device-coherent
// loads.  With many wavefronts it is the racy approximation the thesis runs.
//
// Two variants of the auxiliary sums N_gk, T_gk and B_k (the thesis lets them
// drift during an iteration and corrects them regularly):
//   LIVE   updated with atomics like the other counts; with W = 1 the pass is
//          then exactly sequential collapsed Gibbs (Algorithm SPDP-Full-Gibbs
//          with stored r).  Every token updates one of only G K (and K)
//          counters, so at many wavefronts these atomics serialise.
//   held   the sums keep their sweep-start values during the pass (the token's
//          own contribution removed when it is read) and are regenerated with
//          the counts afterwards; the word, shadow-base and document counts
//          stay live.
//
// Live counts are read past the compute unit's vector cache (agent-scope
// atomic loads), so a wave never sees a line cached before another wave's
// update.  Counts read are clamped to a valid range where races could break
// them (a cell with customers but no table weighs zero).
#include "sampler_common.hpp"

namespace spdp {

namespace {

struct AsyncArgs {
    const int32_t *order;     // [N] visiting order
    const int32_t *tok_doc;   // [N] document of each token
    const int32_t *gw;        // [N] row index g V + w
    const int32_t *doc_group; // [D]
    int32_t *zr;              // [N] state, updated in place
    int32_t *nt;              // [G V][Kp] packed n | t << 16, live
    int32_t *B;               // [V][Kp] shadow-base table counts, live
    int32_t *Ngk, *Tgk;       // [G][Kp] live
    int32_t *Bk;              // [Kp] live
    int32_t *cdk;             // [D][Kp] document-topic counts, live
    const float2 *Q;
    const double *logS;
    int64_t N, nQ;
    int32_t V, K, Kp, ncap;
    uint64_t seed;
    uint32_t sweep;
    float alpha, a, b, gamma, Vgamma;
    double alpha64, a64, b64, gamma64, Vgamma64;
};

__device__ __forceinline__ int32_t coherent_load(const int32_t *p)
{
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// atomic add whose old value the wave waits for (the update has reached the
// device-coherent level before the wave goes on)
__device__ __forceinline__ int32_t add_wait(int32_t *p, int32_t v)
{
    return __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

template <int KPL>
__device__ __forceinline__ void coherent_slice(int32_t (&v)[KPL], const int32_t *row, int32_t kbase,
                                               int32_t Kp)
{
#pragma unroll
    for (int j = 0; j < KPL; ++j) v[j] = (kbase + j < Kp) ? coherent_load(row + kbase + j) : 0;
}

// Relative distance from a CDF boundary below which the fp32 decision is
// re-taken in fp64 (as in the snapshot kernel, with two more roundings for the
// per-token divisions).
constexpr float kAsyncMargin = 1e-5f;

// fp64 weights of topic k from the counts as read (token already removed).
struct Exact2 {
    double w1, w0;
};

__device__ Exact2 exact_async(const AsyncArgs &A, int32_t nt_raw, int32_t b_raw, int32_t c_raw,
                              int32_t N_raw, int32_t T_raw, int32_t Bk_raw)
{
    Exact2 e{0.0, 0.0};
    const int64_t nn = max(nt_raw & kCountMax, 0), tt = nt_raw >> kCountBits;
    double q0, q1;
    if (nn <= 0) {
        q0 = 0.0;
        q1 = 1.0;
    } else if (tt <= 0) {
        return e;
    } else {
        const int64_t n_ = nn < A.ncap ? nn : A.ncap - 1;
        const int64_t t_ = tt > n_ ? n_ : tt;
        const double ls = A.logS[tri_index(n_, t_)];
        q0 = (double)(n_ - t_ + 1) / (double)(n_ + 1) * exp(A.logS[tri_index(n_ + 1, t_)] - ls);
        q1 = (double)(t_ + 1) / (double)(n_ + 1) * exp(A.logS[tri_index(n_ + 1, t_ + 1)] - ls);
    }
    const double doc = A.alpha64 + (double)max(c_raw, 0);
    const double N = (double)max(N_raw, 0), T = (double)max(T_raw, 0);
    e.w0 = doc / (A.b64 + N) * q0;
    e.w1 = doc * (A.b64 + A.a64 * T) / (A.b64 + N) * (A.gamma64 + (double)max(b_raw, 0)) /
           (A.Vgamma64 + (double)max(Bk_raw, 0)) * q1;
    return e;
}

template <int KPL, bool LIVE>
__global__ void __launch_bounds__(64) k_sample_async(AsyncArgs A)
{
    const int32_t lane = threadIdx.x, kbase = lane * KPL;
    const int64_t W = gridDim.x;
    for (int64_t p = blockIdx.x; p < A.N; p += W) {
        const int64_t i = A.order[p];
        const int32_t q = A.gw[i];
        const int32_t d = A.tok_doc[i];
        const int32_t g = A.doc_group[d];
        const int32_t w = q - g * A.V;
        // values every lane must agree on are taken from the first lane
        const int32_t zr0 = __builtin_amdgcn_readfirstlane(coherent_load(A.zr + i));
        const int32_t k0 = zr_topic(zr0), r0 = zr0 & 1;
        const int64_t gK = (int64_t)g * A.Kp;

        // the only head of a cell that keeps other customers stays (point mass)
        const int32_t own =
            __builtin_amdgcn_readfirstlane(coherent_load(A.nt + (int64_t)q * A.Kp + k0));
        if (r0 && (own >> kCountBits) == 1 && (own & kCountMax) > 1) continue;

        // remove the token from the global counts (lane 0), and wait for it
        int32_t sink = 0;
        if (lane == 0) {
            sink += add_wait(A.nt + (int64_t)q * A.Kp + k0, -(1 + (r0 << kCountBits)));
            sink += add_wait(A.cdk + (int64_t)d * A.Kp + k0, -1);
            if (r0) sink += add_wait(A.B + (int64_t)w * A.Kp + k0, -1);
            if constexpr (LIVE) {
                sink += add_wait(A.Ngk + gK + k0, -1);
                if (r0) {
                    sink += add_wait(A.Tgk + gK + k0, -1);
                    sink += add_wait(A.Bk + k0, -1);
                }
            }
        }
        asm volatile("" ::"v"(sink));

        // the counts as they are now
        int32_t n[KPL], bw[KPL], c[KPL], Nk[KPL], Tk[KPL], Bt[KPL];
        coherent_slice<KPL>(n, A.nt + (int64_t)q * A.Kp, kbase, A.Kp);
        coherent_slice<KPL>(bw, A.B + (int64_t)w * A.Kp, kbase, A.Kp);
        coherent_slice<KPL>(c, A.cdk + (int64_t)d * A.Kp, kbase, A.Kp);
        if constexpr (LIVE) {
            coherent_slice<KPL>(Nk, A.Ngk + gK, kbase, A.Kp);
            coherent_slice<KPL>(Tk, A.Tgk + gK, kbase, A.Kp);
            coherent_slice<KPL>(Bt, A.Bk, kbase, A.Kp);
        } else {
            // sweep-start sums (unchanged during the pass): cached loads, the
            // token's own contribution taken out
            load_slice<KPL>(Nk, A.Ngk + gK, kbase, A.Kp);
            load_slice<KPL>(Tk, A.Tgk + gK, kbase, A.Kp);
            load_slice<KPL>(Bt, A.Bk, kbase, A.Kp);
#pragma unroll
            for (int j = 0; j < KPL; ++j) {
                const int32_t own_k = (kbase + j == k0) ? 1 : 0;
                Nk[j] -= own_k;
                Tk[j] -= own_k * r0;
                Bt[j] -= own_k * r0;
            }
        }

        constexpr int NO = 2 * KPL;
        float s[NO];
        float acc = 0.0f;
        const uint32_t q_last = (uint32_t)(A.nQ - 1);
#pragma unroll
        for (int j = 0; j < KPL; ++j) {
            const bool valid = kbase + j < A.K;
            const uint32_t cn = (uint32_t)max(n[j] & kCountMax, 0), ct = (uint32_t)(n[j] >> kCountBits);
            uint32_t ix = ((cn * (cn + 1)) >> 1) + ct;
            ix = ix < q_last ? ix : q_last;
            const float2 qq = A.Q[ix];
            const float doc = A.alpha + (float)max(c[j], 0);
            const float inv = 1.0f / (A.b + (float)max(Nk[j], 0));
            const float f1 = (A.b + A.a * (float)max(Tk[j], 0)) * inv /
                             (A.Vgamma + (float)max(Bt[j], 0));
            const float w1 = valid ? doc * f1 * (A.gamma + (float)max(bw[j], 0)) * qq.y : 0.0f;
            const float w0 = valid ? doc * inv * qq.x : 0.0f;
            acc += w1;
            s[2 * j] = acc;
            acc += w0;
            s[2 * j + 1] = acc;
        }
        const float incl = wave_inclusive_sum(acc);
        const float excl = wave_shift_right(incl);
        const float total = readlane_f(incl, 63);
        const uint32_t xr = philox_x0(A.seed, (uint64_t)i, A.sweep, kPurposeSample);
        const float u = (float)(xr >> 8) * (1.0f / 16777216.0f);
        const float target = u * total;
        const float rel = target - excl;
        int32_t cnt = 0;
#pragma unroll
        for (int j = 0; j < NO; ++j) cnt += (s[j] <= rel) ? 1 : 0;
        const unsigned long long cross = __ballot(cnt < NO);
        int32_t jstar = -1;
        bool fix = true;
        if (cross) {
            const int32_t L = __ffsll((long long)cross) - 1;
            const int32_t cL = readlane(cnt, L);
            const float hi = readlane_f(excl + s[cL], L);
            const float lo = readlane_f(cL > 0 ? excl + s[cL > 0 ? cL - 1 : 0] : excl, L);
            const float margin = kAsyncMargin * total;
            fix = (target - lo < margin) || (hi - target < margin);
            jstar = L * NO + cL;
        }
        if (fix) {
            // fp64 weights from the same counts, fp64 prefix sums, same uniform
            double acc64 = 0.0;
#pragma unroll
            for (int j = 0; j < KPL; ++j) {
                if (kbase + j < A.K) {
                    const Exact2 e = exact_async(A, n[j], bw[j], c[j], Nk[j], Tk[j], Bt[j]);
                    acc64 += e.w1;
                    acc64 += e.w0;
                }
            }
            double incl64 = acc64;
#pragma unroll
            for (int o = 1; o < 64; o <<= 1) {
                const double y = __shfl_up(incl64, o);
                if (lane >= o) incl64 += y;
            }
            double run = __shfl_up(incl64, 1);
            if (lane == 0) run = 0.0;
            const double target64 = (double)u * __shfl(incl64, 63);
            int32_t cand = -1, lastp = -1;
#pragma unroll
            for (int j = 0; j < KPL; ++j) {
                if (kbase + j >= A.K) continue;
                const Exact2 e = exact_async(A, n[j], bw[j], c[j], Nk[j], Tk[j], Bt[j]);
                run += e.w1;
                if (e.w1 > 0.0) {
                    lastp = 2 * j;
                    if (cand < 0 && run > target64) cand = 2 * j;
                }
                run += e.w0;
                if (e.w0 > 0.0) {
                    lastp = 2 * j + 1;
                    if (cand < 0 && run > target64) cand = 2 * j + 1;
                }
            }
            jstar = -1;
            const unsigned long long m2 = __ballot(cand >= 0);
            if (m2) {
                const int32_t L = __ffsll((long long)m2) - 1;
                jstar = L * NO + readlane(cand, L);
            } else {
                const unsigned long long m3 = __ballot(lastp >= 0);
                if (m3) {
                    const int32_t L = 63 - __clzll((long long)m3);
                    jstar = L * NO + readlane(lastp, L);
                }
            }
        }
        // no outcome with weight (possible only under races): keep the state
        const int32_t k1 = jstar >= 0 ? (jstar >> 1) : k0;
        const int32_t r1 = jstar >= 0 ? 1 - (jstar & 1) : r0;

        // add the token at its new cell (lane 0), and wait for it
        if (lane == 0) {
            int32_t sink2 = 0;
            sink2 += add_wait(A.nt + (int64_t)q * A.Kp + k1, 1 + (r1 << kCountBits));
            sink2 += add_wait(A.cdk + (int64_t)d * A.Kp + k1, 1);
            if (r1) sink2 += add_wait(A.B + (int64_t)w * A.Kp + k1, 1);
            if constexpr (LIVE) {
                sink2 += add_wait(A.Ngk + gK + k1, 1);
                if (r1) {
                    sink2 += add_wait(A.Tgk + gK + k1, 1);
                    sink2 += add_wait(A.Bk + k1, 1);
                }
            }
            __hip_atomic_store(A.zr + i, zr_pack(k1, r1), __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
            asm volatile("" ::"v"(sink2));
        }
    }
}

// document-topic counts of the current state: one wave per document
__global__ void __launch_bounds__(64) k_doc_counts(int32_t D, int32_t Kp,
                                                   const int64_t *__restrict__ doc_off,
                                                   const int32_t *__restrict__ zr,
                                                   int32_t *__restrict__ cdk)
{
    __shared__ int32_t h[SPDP_MAX_K];
    const int32_t d = blockIdx.x;
    if (d >= D) return;
    for (int32_t k = threadIdx.x; k < Kp; k += 64) h[k] = 0;
    __syncthreads();
    for (int64_t i = doc_off[d] + threadIdx.x; i < doc_off[d + 1]; i += 64)
        atomicAdd(&h[zr_topic(zr[i])], 1);
    __syncthreads();
    int32_t *row = cdk + (int64_t)d * Kp;
    for (int32_t k = threadIdx.x; k < Kp; k += 64) row[k] = h[k];
}

// token -> document, and the token's position inside its document (the key
// of the visiting order)
__global__ void __launch_bounds__(64) k_tok_doc(int32_t D, const int64_t *__restrict__ doc_off,
                                                int32_t *__restrict__ tok_doc,
                                                int32_t *__restrict__ pos)
{
    const int32_t d = blockIdx.x;
    if (d >= D) return;
    const int64_t beg = doc_off[d];
    for (int64_t i = beg + threadIdx.x; i < doc_off[d + 1]; i += 64) {
        tok_doc[i] = d;
        pos[i] = (int32_t)(i - beg);
    }
}

template <int KPL>
hipError_t launch_async_kpl(const AsyncArgs &A, int32_t waves, bool live, hipStream_t st)
{
    if (live)
        hipLaunchKernelGGL((k_sample_async<KPL, true>), dim3((unsigned)waves), dim3(64), 0, st, A);
    else
        hipLaunchKernelGGL((k_sample_async<KPL, false>), dim3((unsigned)waves), dim3(64), 0, st, A);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_tok_doc(const Model &m, const int64_t *doc_off, int32_t *tok_doc, int32_t *pos,
                          hipStream_t st)
{
    if (m.D <= 0 || m.N <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_tok_doc, dim3((unsigned)m.D), dim3(64), 0, st, m.D, doc_off, tok_doc, pos);
    return hipGetLastError();
}

hipError_t launch_doc_counts(const Model &m, const DeviceBuffers &b, const int32_t *zr,
                             int32_t *cdk, hipStream_t st)
{
    if (m.D <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_doc_counts, dim3((unsigned)m.D), dim3(64), 0, st, m.D, m.Kp, b.doc_off,
                       zr, cdk);
    return hipGetLastError();
}

hipError_t launch_sample_async(const Model &m, const DeviceBuffers &b, const int32_t *order,
                               const int32_t *tok_doc, int32_t *cdk, int32_t *zr, uint32_t sweep,
                               uint64_t seed, int32_t waves, bool live_totals, hipStream_t st)
{
    if (m.D <= 0 || m.N <= 0) return hipSuccess;
    AsyncArgs A;
    A.order = order;
    A.tok_doc = tok_doc;
    A.gw = b.gw;
    A.doc_group = b.doc_group;
    A.zr = zr;
    A.nt = b.nt;
    A.B = b.B;
    A.Ngk = b.Ngk;
    A.Tgk = b.Tgk;
    A.Bk = b.Bk;
    A.cdk = cdk;
    A.Q = b.Q;
    A.logS = b.logS;
    A.N = m.N;
    A.nQ = tri_index(m.ncap, 0);
    A.V = m.V;
    A.K = m.K;
    A.Kp = m.Kp;
    A.ncap = m.ncap;
    A.seed = seed;
    A.sweep = sweep;
    A.alpha = (float)m.alpha;
    A.a = (float)m.a;
    A.b = (float)m.b;
    A.gamma = (float)m.gamma;
    A.Vgamma = (float)((double)m.V * m.gamma);
    A.alpha64 = m.alpha;
    A.a64 = m.a;
    A.b64 = m.b;
    A.gamma64 = m.gamma;
    A.Vgamma64 = (double)m.V * m.gamma;
    switch (sampler_kpl(m.K)) {
    case 1: return launch_async_kpl<1>(A, waves, live_totals, st);
    case 2: return launch_async_kpl<2>(A, waves, live_totals, st);
    case 4: return launch_async_kpl<4>(A, waves, live_totals, st);
    case 8: return launch_async_kpl<8>(A, waves, live_totals, st);
    case 12: return launch_async_kpl<12>(A, waves, live_totals, st);
    default: return launch_async_kpl<16>(A, waves, live_totals, st);
    }
}

}  // namespace spdp
