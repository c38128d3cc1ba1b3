// sample.hip -- the per-sweep resampling kernel (gfx950, wave64).
//
// One wavefront per document.  The shared counts (n, t, B, N_gk, T_gk, B_k)
// are the snapshot of the sweep start and are only read; the document's own
// doc-topic row c[k] is live in LDS and its tokens run in order, so
// documents are independent and the result does not depend on scheduling.
//
// Lane l owns the KPL contiguous topics [l KPL, l KPL + KPL) and, for each
// token, loads its slices of the packed count row (n | t << 16)[g][w][.] and
// of the shadow-base row B[w][.] (coalesced 16-byte loads; the next token's
// rows are in flight while the current token is sampled).  The 2K unnormalised weights of the thesis's
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
    const int32_t *nt;
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
    int64_t nQ;
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
__device__ Exact exact_pair(const SampleArgs &A, int32_t k, int32_t k0, int32_t r0, int32_t nt_raw,
                            int32_t b_raw, int32_t c_raw, const int32_t *Ng, const int32_t *Tg)
{
    Exact e{0.0, 0.0};
    if (k >= A.K) return e;
    const int32_t n_raw = nt_raw & kCountMax, t_raw = nt_raw >> kCountBits;
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

template <int KPL>
__device__ __forceinline__ void lds_slice(float (&v)[KPL], const float *base)
{
    if constexpr (KPL % 4 == 0) {
#pragma unroll
        for (int c = 0; c < KPL / 4; ++c) {
            const float4 x = reinterpret_cast<const float4 *>(base)[c];
            v[4 * c + 0] = x.x;
            v[4 * c + 1] = x.y;
            v[4 * c + 2] = x.z;
            v[4 * c + 3] = x.w;
        }
    } else if constexpr (KPL == 2) {
        const float2 x = *reinterpret_cast<const float2 *>(base);
        v[0] = x.x;
        v[1] = x.y;
    } else {
        v[0] = base[0];
    }
}

template <int KPL, bool TRACE>
__global__ void __launch_bounds__(64, (KPL <= 8 ? 4 : 2)) k_sample(SampleArgs A)
{
    constexpr int NO = 2 * KPL;  // outcomes per lane
    // live document row c[k], the group's per-topic constants f0, f1 and the
    // products a0 = (alpha + c) f0, a1 = (alpha + c) f1 (kept in step with c)
    __shared__ int32_t c_lds[64 * KPL];
    __shared__ float f0_lds[64 * KPL];
    __shared__ float f1_lds[64 * KPL];
    __shared__ __attribute__((aligned(16))) float a0_lds[64 * KPL];
    __shared__ __attribute__((aligned(16))) float a1_lds[64 * KPL];

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
#pragma unroll
    for (int j = 0; j < KPL; ++j) {
        const float doc = A.alpha + (float)c_lds[kbase + j];
        a0_lds[kbase + j] = doc * f0_lds[kbase + j];
        a1_lds[kbase + j] = doc * f1_lds[kbase + j];
    }
    __syncthreads();

    // token stream: 64 tokens per chunk, lane l holds token base + l
    int64_t cbase = beg;
    int32_t gw_c = (beg + lane < end) ? A.gw[beg + lane] : 0;
    int32_t zr_c = (beg + lane < end) ? A.zr_old[beg + lane] : 0;
    int32_t gw_n = 0, zr_n = 0;
    int32_t out_c = 0;
    const uint32_t q_last = (uint32_t)(A.nQ - 1);

    Slice<KPL> rc, rb;  // packed count row and shadow-base row of the current token
    {
        const int32_t q = readlane(gw_c, 0);
        load_slice<KPL>(rc, A.nt + (int64_t)q * A.Kp, kbase, A.Kp);
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
        const int32_t q = readlane(gw_c, idx);
        // the token's own cell and topic totals (uniform loads)
        const int32_t nt0 = A.nt[(int64_t)q * A.Kp + k0];
        const int32_t b0 = A.B[(int64_t)(q - gV) * A.Kp + k0];
        const int32_t N0 = Ng[k0], T0 = Tg[k0], Bk0 = A.Bk[k0];
        const int32_t n0 = nt0 & kCountMax, t0 = nt0 >> kCountBits;
        // only head of a cell that keeps other customers: point mass
        const bool sole = r0 && t0 == 1 && n0 > 1;

        // Stirling ratio pairs of every topic's cell as it stands (the token's
        // own topic is recomputed below with the token removed); gathered
        // before the next token's rows are requested
        float2 qv[KPL];
#pragma unroll
        for (int j = 0; j < KPL; ++j) {
            const uint32_t cn = (uint32_t)rc.v[j] & kCountMax;
            const uint32_t ct = (uint32_t)rc.v[j] >> kCountBits;
            uint32_t ix = ((cn * (cn + 1)) >> 1) + ct;
            ix = ix < q_last ? ix : q_last;
            qv[j] = A.Q[ix];
        }

        // next token's rows
        Slice<KPL> xc, xb;
        const bool have_next = (i + 1 < end);
        if (have_next) {
            const int32_t q1 = (idx + 1 < 64) ? readlane(gw_c, idx + 1) : readlane(gw_n, 0);
            load_slice<KPL>(xc, A.nt + (int64_t)q1 * A.Kp, kbase, A.Kp);
            load_slice<KPL>(xb, A.B + (int64_t)(q1 - gV) * A.Kp, kbase, A.Kp);
        }

        int32_t result = zr0;
        float u = -1.0f;
        if (!sole) {
            // the token's own topic with the token removed: fp64 constants
            // rounded once, as for the other topics
            const int32_t n0r = n0 - 1, t0r = t0 - r0;
            uint32_t ix0 = (uint32_t)(((n0r * (n0r + 1)) >> 1) + t0r);
            ix0 = ix0 < q_last ? ix0 : q_last;
            const float2 q0v = A.Q[ix0];
            const int32_t c0 = c_lds[k0];
            const double inv = 1.0 / (A.b + (double)(N0 - 1));
            const float f0k = (float)inv;
            const float f1k =
                (float)((A.b + A.a * (double)(T0 - r0)) * inv / (A.Vgamma + (double)(Bk0 - r0)));
            const float doc0 = A.alpha + (float)(c0 - 1);
            const float w1k0 = doc0 * f1k * (A.gamma + (float)(b0 - r0)) * q0v.y;
            const float w0k0 = doc0 * f0k * q0v.x;

            // weights and lane-local inclusive prefix sums
            float a0[KPL], a1[KPL];
            lds_slice<KPL>(a0, a0_lds + kbase);
            lds_slice<KPL>(a1, a1_lds + kbase);
            float s[NO];
            float acc = 0.0f;
#pragma unroll
            for (int j = 0; j < KPL; ++j) {
                const bool own = (kbase + j == k0);
                const float bw = A.gamma + (float)rb.v[j];
                float w1 = a1[j] * bw * qv[j].y;
                float w0 = a0[j] * qv[j].x;
                w1 = own ? w1k0 : w1;
                w0 = own ? w0k0 : w0;
                if constexpr (TRACE) {
                    if (i >= A.tr_begin && i < A.tr_end && kbase + j < A.K) {
                        float *o = A.tr_w + (i - A.tr_begin) * 2 * (int64_t)A.K + 2 * (kbase + j);
                        o[0] = w1;
                        o[1] = w0;
                    }
                }
                acc += w1;
                s[2 * j] = acc;
                acc += w0;
                s[2 * j + 1] = acc;
            }
            const float incl = wave_inclusive_sum(acc);
            const float excl = wave_shift_right(incl);
            const float total = readlane_f(incl, 63);

            const uint32_t x = philox_x0(A.seed, (uint64_t)i, A.sweep, kPurposeSample);
            u = (float)(x >> 8) * (1.0f / 16777216.0f);
            const float target = u * total;

            // count the prefixes at or below the target (prefixes are
            // monotone, so the first crossing of this lane is outcome cnt) and
            // flag any prefix within rounding distance of the target
            const float rel = target - excl;
            const float margin = kFixMargin * total;
            int32_t cnt = 0;
            bool near = false;
#pragma unroll
            for (int j = 0; j < NO; ++j) {
                const float dlt = s[j] - rel;
                cnt += (dlt <= 0.0f) ? 1 : 0;
                near |= (fabsf(dlt) < margin);
            }
            const unsigned long long cross = __ballot(cnt < NO);
            int32_t jstar = -1;
            if (cross && !__any(near)) {
                const int32_t L = __ffsll((long long)cross) - 1;
                jstar = L * NO + readlane(cnt, L);
            } else {
                // The draw is within rounding distance of a CDF boundary (or the
                // fp32 scan found no crossing): take it again with fp64 weights
                // from the integer counts, fp64 prefix sums and the same uniform
                // (rolled loops re-reading the current rows from memory keep
                // this rare path from raising the kernel's register count).
                const int32_t *__restrict__ crow = A.nt + (int64_t)q * A.Kp;
                const int32_t *__restrict__ brow = A.B + (int64_t)(q - gV) * A.Kp;
                double acc64 = 0.0;
#pragma unroll 1
                for (int j = 0; j < KPL; ++j) {
                    const int32_t k = kbase + j;
                    if (k >= A.K) break;
                    const Exact e = exact_pair<KPL>(A, k, k0, r0, crow[k], brow[k], c_lds[k],
                                                    Ng, Tg);
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
                    const Exact e = exact_pair<KPL>(A, k, k0, r0, crow[k], brow[k], c_lds[k],
                                                    Ng, Tg);
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
                // token's reads of the LDS rows see this update
                if (lane == 0 && k1 != k0) {
                    const int32_t ca = c_lds[k0] - 1, cb = c_lds[k1] + 1;
                    c_lds[k0] = ca;
                    c_lds[k1] = cb;
                    const float da = A.alpha + (float)ca, db = A.alpha + (float)cb;
                    a0_lds[k0] = da * f0_lds[k0];
                    a1_lds[k0] = da * f1_lds[k0];
                    a0_lds[k1] = db * f0_lds[k1];
                    a1_lds[k1] = db * f1_lds[k1];
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
            rc = xc;
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
    A.nt = b.nt;
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
    A.nQ = tri_index(m.ncap, 0);
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
