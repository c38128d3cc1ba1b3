// sample.hip -- the per-sweep resampling kernel (gfx950, wave64).
//
// One wavefront per document.  The shared counts (n, t, B, N_gk, T_gk, B_k)
// are the snapshot of the sweep start and are only read; the document's own
// doc-topic row c[k] is live in LDS and its tokens run in order, so
// documents are independent and the result does not depend on scheduling.
//
// Lane l owns the KPL contiguous topics [l KPL, l KPL + KPL) and, for each
// token, loads its slices of the rows n[g][w][.], t[g][w][.], B[w][.]
// (coalesced 16-byte loads; the next token's rows are in flight while the
// current token is sampled).  The 2K unnormalised weights of the thesis's
// conditionals (Eq. SPDP-sampling-w-z-r0 / -r1, P = I), with the token
// removed from its own cell:
//   W(k, r=1) = (alpha + c'_k) f1[g][k] (gamma + B'_wk) Q1(n', t')
//   W(k, r=0) = (alpha + c'_k) f0[g][k] Q0(n', t')
// where f0 = 1/(b + N'), f1 = (b + a T')/(b + N')/(V gamma + B'_k) are the
// per-(group, topic) sweep constants (recomputed in fp64 for the token's own
// topic) and (Q0, Q1) the folded Stirling ratios.  Outcome j = 2k is (k, r=1),
// j = 2k+1 is (k, r=0); the lane-local inclusive prefix sums plus a wave scan
// of the lane totals give the CDF, and the draw is the first outcome whose
// prefix exceeds u * total, u the 24-bit Philox uniform of the token.
#include "spdp_internal.hpp"

namespace spdp {

namespace {

struct SampleArgs {
    const int32_t *gw;
    const int64_t *doc_off;
    const int32_t *doc_group;
    const int32_t *zr_old;
    int32_t *zr_new;
    const int32_t *n;
    const int32_t *t;
    const int32_t *B;
    const int32_t *Ngk;
    const int32_t *Tgk;
    const int32_t *Bk;
    const float *f0;
    const float *f1;
    const float2 *Q;
    const double *logS;
    float *tr_w;
    float *tr_u;
    int64_t tr_begin, tr_end;
    uint64_t seed;
    int32_t D, V, K, Kp, ncap;
    int32_t docs_per_xcd;
    uint32_t sweep;
    float alpha, gamma;
    double alpha_d, gamma_d, a, b, Vgamma;
};

// KPL consecutive int32 of one row, loaded with the widest aligned vector
// loads; chunks that start at or beyond the row length are zero.
template <int KPL>
struct Slice {
    int32_t v[KPL];
};

template <int KPL>
__device__ __forceinline__ void load_slice(Slice<KPL> &s, const int32_t *__restrict__ row,
                                           int32_t kbase, int32_t Kp)
{
    if constexpr (KPL % 4 == 0) {
#pragma unroll
        for (int c = 0; c < KPL / 4; ++c) {
            int4 x = make_int4(0, 0, 0, 0);
            if (kbase + 4 * c < Kp) x = *reinterpret_cast<const int4 *>(row + kbase + 4 * c);
            s.v[4 * c + 0] = x.x;
            s.v[4 * c + 1] = x.y;
            s.v[4 * c + 2] = x.z;
            s.v[4 * c + 3] = x.w;
        }
    } else if constexpr (KPL == 2) {
        int2 x = make_int2(0, 0);
        if (kbase < Kp) x = *reinterpret_cast<const int2 *>(row + kbase);
        s.v[0] = x.x;
        s.v[1] = x.y;
    } else {
        static_assert(KPL == 1, "KPL must be 1, 2 or a multiple of 4");
        s.v[0] = (kbase < Kp) ? row[kbase] : 0;
    }
}

template <int KPL>
__device__ __forceinline__ void load_slice_f(float (&s)[KPL], const float *__restrict__ row,
                                             int32_t kbase, int32_t Kp)
{
    Slice<KPL> tmp;
    load_slice<KPL>(tmp, reinterpret_cast<const int32_t *>(row), kbase, Kp);
#pragma unroll
    for (int j = 0; j < KPL; ++j) s[j] = __int_as_float(tmp.v[j]);
}

__device__ __forceinline__ int32_t readlane(int32_t x, int32_t lane)
{
    return __builtin_amdgcn_readlane(x, lane);
}

__device__ __forceinline__ float readlane_f(float x, int32_t lane)
{
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), lane));
}

// Relative distance from a CDF boundary below which the fp32 decision is
// re-taken in fp64.  The fp32 prefix sums are within about 3e-6 of the exact
// ones (at most 7 roundings per weight, at most 2 KPL + 6 additions per
// prefix, KPL <= 16), so outside this margin both decisions agree.
constexpr float kFixMargin = 8e-6f;

// fp64 weights of outcome pair j of this lane, evaluated directly from the
// integer counts and the fp64 log Stirling table (the rare boundary path).
struct Exact {
    double w1, w0;
};

template <int KPL>
__device__ Exact exact_pair(const SampleArgs &A, int32_t k, int32_t k0, int32_t r0, int32_t n_raw,
                            int32_t t_raw, int32_t b_raw, int32_t c_raw, const int32_t *Ng,
                            const int32_t *Tg)
{
    Exact e{0.0, 0.0};
    if (k >= A.K) return e;
    const int32_t del = (k == k0) ? 1 : 0;
    const int64_t nn = n_raw - del, tt = t_raw - del * r0;
    const double bw = (double)(b_raw - del * r0);
    const double N = (double)(Ng[k] - del), T = (double)(Tg[k] - del * r0);
    const double Bt = (double)(A.Bk[k] - del * r0);
    const double doc = (double)A.alpha_d + (double)(c_raw - del);
    double q0, q1;
    if (nn <= 0) {
        q0 = 0.0;
        q1 = 1.0;
    } else {
        const int64_t n_ = nn < A.ncap ? nn : A.ncap - 1;
        const int64_t t_ = tt < 0 ? 0 : (tt > n_ ? n_ : tt);
        const double ls = A.logS[tri_index(n_, t_)];
        q0 = (double)(n_ - t_ + 1) / (double)(n_ + 1) * exp(A.logS[tri_index(n_ + 1, t_)] - ls);
        q1 = (double)(t_ + 1) / (double)(n_ + 1) * exp(A.logS[tri_index(n_ + 1, t_ + 1)] - ls);
    }
    e.w0 = doc / (A.b + N) * q0;
    e.w1 = doc * (A.b + A.a * T) / (A.b + N) * ((double)A.gamma_d + bw) / (A.Vgamma + Bt) * q1;
    return e;
}

template <int KPL, bool TRACE>
__global__ void __launch_bounds__(64, (KPL <= 8 ? 4 : 2)) k_sample(SampleArgs A)
{
    constexpr int NO = 2 * KPL;  // outcomes per lane
    // live document row c[k] and the per-(g, k) constants of the document's group
    __shared__ int32_t c_lds[64 * KPL];
    __shared__ float f0_lds[64 * KPL];
    __shared__ float f1_lds[64 * KPL];

    // blocks are dealt round-robin over the 8 XCDs; give each XCD a
    // contiguous range of documents so a group's hot rows stay in its L2
    const int32_t b = blockIdx.x;
    const int32_t d = (b & 7) * A.docs_per_xcd + (b >> 3);
    if (d >= A.D) return;
    const int64_t beg = A.doc_off[d], end = A.doc_off[d + 1];
    if (beg >= end) return;
    const int32_t lane = threadIdx.x;
    const int32_t g = A.doc_group[d];
    const int32_t kbase = lane * KPL;
    const int32_t gV = g * A.V;
    const int32_t *__restrict__ Ng = A.Ngk + (int64_t)g * A.Kp;
    const int32_t *__restrict__ Tg = A.Tgk + (int64_t)g * A.Kp;

    {
        float f0[KPL], f1[KPL];
        load_slice_f<KPL>(f0, A.f0 + (int64_t)g * A.Kp, kbase, A.Kp);
        load_slice_f<KPL>(f1, A.f1 + (int64_t)g * A.Kp, kbase, A.Kp);
#pragma unroll
        for (int j = 0; j < KPL; ++j) {
            c_lds[kbase + j] = 0;
            f0_lds[kbase + j] = f0[j];
            f1_lds[kbase + j] = f1[j];
        }
    }
    __syncthreads();
    for (int64_t i = beg + lane; i < end; i += 64) atomicAdd(&c_lds[A.zr_old[i] >> 1], 1);
    __syncthreads();

    // token stream: 64 tokens per chunk, lane l holds token base + l
    int64_t cbase = beg;
    int32_t gw_c = (beg + lane < end) ? A.gw[beg + lane] : 0;
    int32_t zr_c = (beg + lane < end) ? A.zr_old[beg + lane] : 0;
    int32_t gw_n = 0, zr_n = 0;
    int32_t out_c = 0;

    Slice<KPL> rn, rt, rb;  // rows of the current token
    {
        const int32_t q = readlane(gw_c, 0);
        load_slice<KPL>(rn, A.n + (int64_t)q * A.Kp, kbase, A.Kp);
        load_slice<KPL>(rt, A.t + (int64_t)q * A.Kp, kbase, A.Kp);
        load_slice<KPL>(rb, A.B + (int64_t)(q - gV) * A.Kp, kbase, A.Kp);
    }

    for (int64_t i = beg; i < end; ++i) {
        const int32_t idx = (int32_t)(i - cbase);
        if (idx == 0 && cbase + 64 < end) {
            // next chunk of the token stream
            gw_n = (cbase + 64 + lane < end) ? A.gw[cbase + 64 + lane] : 0;
            zr_n = (cbase + 64 + lane < end) ? A.zr_old[cbase + 64 + lane] : 0;
        }
        const int32_t zr0 = readlane(zr_c, idx);
        const int32_t k0 = zr0 >> 1, r0 = zr0 & 1;
        // totals of the token's own topic (uniform loads)
        const int32_t N0 = Ng[k0], T0 = Tg[k0], B0 = A.Bk[k0];

        // removal-corrected state of the token's own cell and the Stirling
        // ratio pairs (gathered before the next token's rows are requested)
        float2 qv[KPL];
        bool sole = false;
#pragma unroll
        for (int j = 0; j < KPL; ++j) {
            const int32_t del = (kbase + j == k0) ? 1 : 0;
            if (del && r0 && rt.v[j] == 1 && rn.v[j] > 1) sole = true;
            int32_t a_n = rn.v[j] - del;
            a_n = a_n < 0 ? 0 : (a_n >= A.ncap ? A.ncap - 1 : a_n);
            int32_t a_t = rt.v[j] - del * r0;
            a_t = a_t < 0 ? 0 : (a_t > a_n ? a_n : a_t);
            qv[j] = (a_n == 0) ? make_float2(0.0f, 1.0f)
                               : A.Q[(int64_t)a_n * (a_n + 1) / 2 + a_t];
        }

        // next token's rows
        Slice<KPL> xn, xt, xb;
        const bool have_next = (i + 1 < end);
        if (have_next) {
            const int32_t q1 = (idx + 1 < 64) ? readlane(gw_c, idx + 1) : readlane(gw_n, 0);
            load_slice<KPL>(xn, A.n + (int64_t)q1 * A.Kp, kbase, A.Kp);
            load_slice<KPL>(xt, A.t + (int64_t)q1 * A.Kp, kbase, A.Kp);
            load_slice<KPL>(xb, A.B + (int64_t)(q1 - gV) * A.Kp, kbase, A.Kp);
        }

        int32_t result = zr0;
        float u = -1.0f;
        if (!__any(sole)) {
            // constants of the token's own topic with the token removed (fp64,
            // rounded once, as for the other topics)
            const double inv = 1.0 / (A.b + (double)(N0 - 1));
            const float f0k = (float)inv;
            const float f1k =
                (float)((A.b + A.a * (double)(T0 - r0)) * inv / (A.Vgamma + (double)(B0 - r0)));
            // weights and lane-local inclusive prefix sums
            float s[NO];
            float acc = 0.0f;
#pragma unroll
            for (int j = 0; j < KPL; ++j) {
                const int32_t k = kbase + j;
                const int32_t del = (k == k0) ? 1 : 0;
                const float doc = A.alpha + (float)(c_lds[k] - del);
                const float bw = A.gamma + (float)(rb.v[j] - del * r0);
                const float w1 = doc * (del ? f1k : f1_lds[k]) * bw * qv[j].y;
                const float w0 = doc * (del ? f0k : f0_lds[k]) * qv[j].x;
                if constexpr (TRACE) {
                    if (i >= A.tr_begin && i < A.tr_end && k < A.K) {
                        float *o = A.tr_w + (i - A.tr_begin) * 2 * (int64_t)A.K + 2 * k;
                        o[0] = w1;
                        o[1] = w0;
                    }
                }
                acc += w1;
                s[2 * j] = acc;
                acc += w0;
                s[2 * j + 1] = acc;
            }
            // wave inclusive scan of the lane totals
            float incl = acc;
#pragma unroll
            for (int o = 1; o < 64; o <<= 1) {
                const float y = __shfl_up(incl, o);
                if (lane >= o) incl += y;
            }
            float excl = __shfl_up(incl, 1);
            if (lane == 0) excl = 0.0f;
            const float total = __shfl(incl, 63);

            const uint32_t x = philox_x0(A.seed, (uint64_t)i, A.sweep, kPurposeSample);
            u = (float)(x >> 8) * (1.0f / 16777216.0f);
            const float target = u * total;

            // first outcome whose prefix exceeds the target; an outcome of zero
            // weight can only be first at a lane's start (s[0] == 0), so the
            // guard is needed there only
            int32_t cand = -1;
            float lo = 0.0f, hi = 0.0f;
#pragma unroll
            for (int j = NO - 1; j >= 0; --j) {
                const bool pos = (j == 0) ? (s[0] > 0.0f) : (s[j] > s[j - 1]);
                if (pos && excl + s[j] > target) {
                    cand = j;
                    hi = excl + s[j];
                    lo = excl + (j == 0 ? 0.0f : s[j - 1]);
                }
            }
            int32_t jstar = -1;
            bool fix = true;
            const unsigned long long m1 = __ballot(cand >= 0);
            if (m1) {
                const int32_t L = __ffsll((long long)m1) - 1;
                jstar = L * NO + readlane(cand, L);
                const float margin = kFixMargin * total;
                fix = (target - readlane_f(lo, L) < margin) || (readlane_f(hi, L) - target < margin);
            }
            if (fix) {
                // The draw is within rounding distance of a CDF boundary (or the
                // fp32 scan found no crossing): take it again with fp64 weights
                // from the integer counts, fp64 prefix sums and the same uniform.
                // (rolled loops re-reading the current rows from memory keep
                // this rare path from raising the kernel's register count)
                const int64_t qrow = (int64_t)readlane(gw_c, idx);
                const int32_t *__restrict__ nrow = A.n + qrow * A.Kp;
                const int32_t *__restrict__ trow = A.t + qrow * A.Kp;
                const int32_t *__restrict__ brow = A.B + (qrow - gV) * A.Kp;
                double acc64 = 0.0;
#pragma unroll 1
                for (int j = 0; j < KPL; ++j) {
                    const int32_t k = kbase + j;
                    if (k >= A.K) break;
                    const Exact e = exact_pair<KPL>(A, k, k0, r0, nrow[k], trow[k], brow[k],
                                                    c_lds[k], Ng, Tg);
                    acc64 += e.w1;
                    acc64 += e.w0;
                }
                double incl64 = acc64;
#pragma unroll
                for (int o = 1; o < 64; o <<= 1) {
                    const double y = __shfl_up(incl64, o);
                    if (lane >= o) incl64 += y;
                }
                double run = __shfl_up(incl64, 1);
                if (lane == 0) run = 0.0;
                const double total64 = __shfl(incl64, 63);
                const double target64 = (double)u * total64;
                int32_t cand64 = -1, last64 = -1;
#pragma unroll 1
                for (int j = 0; j < KPL; ++j) {
                    const int32_t k = kbase + j;
                    if (k >= A.K) break;
                    const Exact e = exact_pair<KPL>(A, k, k0, r0, nrow[k], trow[k], brow[k],
                                                    c_lds[k], Ng, Tg);
                    run += e.w1;
                    if (e.w1 > 0.0) {
                        last64 = 2 * j;
                        if (cand64 < 0 && run > target64) cand64 = 2 * j;
                    }
                    run += e.w0;
                    if (e.w0 > 0.0) {
                        last64 = 2 * j + 1;
                        if (cand64 < 0 && run > target64) cand64 = 2 * j + 1;
                    }
                }
                const unsigned long long m2 = __ballot(cand64 >= 0);
                if (m2) {
                    const int32_t L = __ffsll((long long)m2) - 1;
                    jstar = L * NO + readlane(cand64, L);
                } else {
                    const unsigned long long m3 = __ballot(last64 >= 0);
                    if (m3) {
                        const int32_t L = 63 - __clzll((long long)m3);
                        jstar = L * NO + readlane(last64, L);
                    }
                }
            }
            if (jstar >= 0) {
                const int32_t k1 = jstar >> 1, r1 = 1 - (jstar & 1);
                result = zr_pack(k1, r1);
                // DS operations of one wave execute in order, so the next
                // token's reads of c_lds see this update
                if (lane == 0) {
                    c_lds[k0] -= 1;
                    c_lds[k1] += 1;
                }
            }
        }
        if constexpr (TRACE) {
            if (lane == 0 && i >= A.tr_begin && i < A.tr_end) A.tr_u[i - A.tr_begin] = u;
        }

        // buffer the result; write 64 tokens at a time
        if (lane == idx) out_c = result;
        if (idx == 63 || i + 1 == end) {
            if (lane <= idx) A.zr_new[cbase + lane] = out_c;
        }
        if (idx == 63) {
            cbase += 64;
            gw_c = gw_n;
            zr_c = zr_n;
        }
        if (have_next) {
            rn = xn;
            rt = xt;
            rb = xb;
        }
    }
}

template <int KPL>
hipError_t launch_kpl(const SampleArgs &A, bool trace, hipStream_t st)
{
    const unsigned grid = (unsigned)(8 * A.docs_per_xcd);
    if (trace)
        hipLaunchKernelGGL((k_sample<KPL, true>), dim3(grid), dim3(64), 0, st, A);
    else
        hipLaunchKernelGGL((k_sample<KPL, false>), dim3(grid), dim3(64), 0, st, A);
    return hipGetLastError();
}

}  // namespace

int sampler_kpl(int32_t K)
{
    if (K <= 64) return 1;
    if (K <= 128) return 2;
    if (K <= 256) return 4;
    if (K <= 512) return 8;
    if (K <= 768) return 12;
    return 16;
}

int32_t padded_K(int32_t K)
{
    const int kpl = sampler_kpl(K);
    const int align = kpl >= 4 ? 4 : kpl;
    return (K + align - 1) / align * align;
}

hipError_t launch_sample(const Model &m, const DeviceBuffers &b, const int32_t *zr_old,
                         int32_t *zr_new, uint32_t sweep, uint64_t seed, float *tr_w, float *tr_u,
                         int64_t tr_begin, int64_t tr_end, hipStream_t st)
{
    if (m.D <= 0 || m.N <= 0) return hipSuccess;
    SampleArgs A;
    A.gw = b.gw;
    A.doc_off = b.doc_off;
    A.doc_group = b.doc_group;
    A.zr_old = zr_old;
    A.zr_new = zr_new;
    A.n = b.n;
    A.t = b.t;
    A.B = b.B;
    A.Ngk = b.Ngk;
    A.Tgk = b.Tgk;
    A.Bk = b.Bk;
    A.f0 = b.f0;
    A.f1 = b.f1;
    A.Q = b.Q;
    A.logS = b.logS;
    A.tr_w = tr_w;
    A.tr_u = tr_u;
    A.tr_begin = tr_begin;
    A.tr_end = tr_end;
    A.seed = seed;
    A.D = m.D;
    A.V = m.V;
    A.K = m.K;
    A.Kp = m.Kp;
    A.ncap = m.ncap;
    A.docs_per_xcd = (m.D + 7) / 8;
    A.sweep = sweep;
    A.alpha = (float)m.alpha;
    A.gamma = (float)m.gamma;
    A.alpha_d = m.alpha;
    A.gamma_d = m.gamma;
    A.a = m.a;
    A.b = m.b;
    A.Vgamma = (double)m.V * m.gamma;
    const bool trace = (tr_w != nullptr);
    switch (sampler_kpl(m.K)) {
    case 1: return launch_kpl<1>(A, trace, st);
    case 2: return launch_kpl<2>(A, trace, st);
    case 4: return launch_kpl<4>(A, trace, st);
    case 8: return launch_kpl<8>(A, trace, st);
    case 12: return launch_kpl<12>(A, trace, st);
    default: return launch_kpl<16>(A, trace, st);
    }
}

}  // namespace spdp
