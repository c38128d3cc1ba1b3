// sample.hip -- the per-sweep resampling kernel (gfx950, wave64).
//
// One wavefront per document.  The shared counts (n, t, B, N_gk, T_gk, B_k)
// are the snapshot of the sweep start and are only read; the document's own
// doc-topic row c[k] is live in LDS and its tokens run in order, so
// documents are independent and the result does not depend on scheduling.
//
// Lane l owns the KPL contiguous topics [l KPL, l KPL + KPL).  For each token
// the wave loads its packed count row (n | t << 16)[g][w][.] -- or, for a
// (group, word) pair with at most 255 tokens, the row's 16-bit copy
// (n | t << 8), half the bytes -- and its
// shadow-base row B[w][.] with coalesced vector loads, two tokens ahead of
// use (three register sets rotate, so no copy ever waits on a load in
// flight), and gathers the folded Stirling ratios (Q0, Q1) of every cell.  The
// 2K unnormalised weights of the thesis's conditionals (Eq.
// SPDP-sampling-w-z-r0 / -r1, P = I), with the token removed from its own
// cell, are
//   W(k, r=1) = (alpha + c'_k) f1[g][k] (gamma + B'_wk) Q1(n', t')
//   W(k, r=0) = (alpha + c'_k) f0[g][k] Q0(n', t')
// with f0 = 1/(b + N'), f1 = (b + a T')/(b + N')/(V gamma + B'_k) the
// per-(group, topic) sweep constants, taken for the token's own topic from
// the removed-customer table fk.  Outcome j = 2k is (k, r=1), j = 2k+1 is
// (k, r=0); the lane-local inclusive prefix sums plus a wave scan of the lane
// totals give the CDF, and the draw is the first outcome whose prefix exceeds
// u * total, u the 24-bit Philox uniform of the token.  A draw within fp32
// rounding distance of a CDF boundary is taken again in fp64.
#include "sampler_common.hpp"

namespace spdp {

namespace {

struct SampleArgs {
    const int32_t *gw;
    const int64_t *doc_off;
    const int32_t *doc_group;
    const int32_t *zr_old;
    int32_t *zr_new;
    const int32_t *nt;
    const uint16_t *nt16;
    const uint8_t *tok_narrow;
    const int32_t *B;
    const uint16_t *B16;
    const int32_t *wide;
    int32_t *claim;  // [9] documents claimed per XCD by the persistent launch, and the
                     // workgroups of that launch that have finished (zero between launches)
    const float *f0;
    const float *f1;
    const float *fk;
    const float2 *Q;
    const ExactCtx *exact;
    float *tr_w;
    float *tr_u;
    int64_t tr_begin, tr_end;
    uint64_t seed;
    int32_t D, V, K, Kp;
    int64_t nQ, GK;
    int32_t docs_per_xcd;
    uint32_t sweep;
    float alpha, gamma;
};

// Tokens per step of the token stream.  The stream registers hold 64 tokens
// (lane l: token base + l); advancing by 48 leaves the next two tokens of
// every position in the same registers, and 48 is a multiple of the three
// rotating row buffers.
constexpr int32_t kChunk = 48;

// Distance from a CDF boundary, as a fraction of the total, below which the
// fp32 decision is taken again in fp64.  To first order in u = 2^-24 against
// exact arithmetic: every fp32 weight carries at most 9 relative roundings
// (alpha, gamma, the per-topic constant and the ratio pair each rounded once
// from fp64, the two sums with counts, three products), which moves the
// target's distance to any boundary by at most 9u of the total; the
// summation of a boundary (2 KPL - 1 lane-local additions, 6 in the wave
// scan) and of the total behind the target each add at most (2 KPL + 5)u;
// the target's product, its lane offset, the compared boundary and the
// distance itself one rounding each.  So the fp32 distance is within
// (4 KPL + 23)u of the exact one, and outside (4 KPL + 32)u both decisions
// agree.
template <int KPL>
__device__ __forceinline__ float fix_margin()
{
    return (float)(4 * KPL + 32) * 5.97e-8f;
}

// fp64 weights of outcome pair k, evaluated directly from the integer counts
// and the fp64 ratio pairs (the rare boundary path).
struct Exact {
    double w1, w0;
};

__device__ Exact exact_pair(const ExactCtx &A, int32_t k, int32_t k0, int32_t r0, int32_t nt_raw,
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
    const double doc = A.alpha + (double)(c_raw - del);
    const double2 qq = A.Q64[exact_q_index(A, (int32_t)nn, (int32_t)tt)];
    const double q0 = qq.x, q1 = qq.y;
    e.w0 = doc / (A.b + N) * q0;
    e.w1 = doc * (A.b + A.a * T) / (A.b + N) * (A.gamma + bw) / (A.Vgamma + Bt) * q1;
    return e;
}

// The rows one token needs: this lane's slices of its packed count row and
// of the 16-bit copy of its shadow-base row, min(B, 65535).
template <int KPL>
struct Rows {
    static constexpr int NB = (KPL + 1) / 2;
    int32_t n[KPL];
    uint32_t bw[NB];  // shadow-base counts, two 16-bit ones per word
    __device__ __forceinline__ int32_t b(int j) const
    {
        return (int32_t)((bw[j >> 1] >> (16 * (j & 1))) & 0xFFFFu);
    }
    // the same for a wave-uniform j that is not a compile-time constant
    __device__ __forceinline__ int32_t b_at(int j) const
    {
        return (int32_t)((pick(bw, j >> 1) >> (16 * (j & 1))) & 0xFFFFu);
    }
};

// Per-wave state of one document.
template <int KPL>
struct DocWave {
    int32_t lane, kbase, gV;
    int64_t gK, cb, end;
    int32_t *c_lds;
    float *f0_lds, *f1_lds, *a0_lds, *a1_lds;
    // token stream: lane l holds the row index, packed state, narrow-row flag
    // and uniform of token cb + l (lanes past the document's end repeat its
    // last token)
    int32_t gw_c, zr_c, nar_c, out_c;
    float u_c;
};

template <int KPL>
__device__ __forceinline__ void load_rows(const SampleArgs &A, const DocWave<KPL> &W, int32_t x,
                                          Rows<KPL> &R)
{
    const int32_t q = readlane(W.gw_c, x);
    const int64_t wrow = (int64_t)(q - W.gV) * A.Kp;
    // a narrow row as its 16-bit copy (half the bytes), widened at use
    load_count_row<KPL>(R.n, A.nt, A.nt16, q, W.kbase, A.Kp, readlane(W.nar_c, x) != 0);
    load_half_row<KPL>(R.bw, A.B16 + wrow, W.kbase, A.Kp);
}

// Shadow-base count of this lane's slot j for the fp64 path: in the 32-bit
// launch a saturated 16-bit cell is read from B itself.
template <int KPL, bool WIDE>
__device__ __forceinline__ int32_t exact_b(const SampleArgs &A, const DocWave<KPL> &W, int32_t x,
                                           const Rows<KPL> &R, int j)
{
    int32_t v = R.b_at(j);
    if constexpr (WIDE) {
        if (v == 0xFFFF) v = A.B[(int64_t)(readlane(W.gw_c, x) - W.gV) * A.Kp + W.kbase + j];
    }
    return v;
}

// Stream registers of the tokens from W.cb on (lanes past the document's end
// repeat its last token), and the tokens' uniforms: Philox word 0 at counter
// (token lo, token hi, sweep, 0), one token per lane, so the rounds run on the
// vector unit once per 48 tokens.  The loads are waited for here, so that no
// token's wait on its prefetched rows has to cover them.
template <int KPL>
__device__ __forceinline__ void load_stream(const SampleArgs &A, DocWave<KPL> &W, int64_t last)
{
    const int64_t t = min(W.cb + W.lane, last);
    W.gw_c = A.gw[t];
    W.zr_c = A.zr_old[t];
    W.nar_c = A.tok_narrow[t];
    const uint32_t xr = philox_x0(A.seed, (uint64_t)(W.cb + W.lane), A.sweep, kPurposeSample);
    W.u_c = (float)(xr >> 8) * (1.0f / 16777216.0f);
    asm volatile("" ::"v"(W.gw_c), "v"(W.zr_c), "v"(W.nar_c));
}

// Token cb + x: sample it with the rows in `cur` and request the rows of the
// token two places ahead into `fill`.
template <int KPL, bool TRACE, bool WIDE, bool BIGQ>
__device__ __forceinline__ void sample_token(const SampleArgs &A, DocWave<KPL> &W, int32_t x,
                                             Rows<KPL> &cur, Rows<KPL> &fill)
{
    constexpr int NO = 2 * KPL;  // outcomes per lane
    const int32_t lane = W.lane, kbase = W.kbase;
    const int64_t i = W.cb + x;
    // Wave priorities: the part of a token that issues its loads (the ratio
    // gathers and the rows two tokens ahead) runs at priority 2 and the serial
    // scan and draw at 3, above the weight loops (priority 0) of the other
    // wavefronts on the SIMD, so that a wavefront's loads leave and its draw
    // resolves without queueing behind their vector work.
    __builtin_amdgcn_s_setprio(2);
    if (readlane(W.nar_c, x)) widen_cells<KPL>(cur.n, kbase);

    const int32_t zr0 = readlane(W.zr_c, x);
    const int32_t k0 = zr0 >> 1, r0 = zr0 & 1;
    const uint32_t q_last = (uint32_t)(A.nQ - 1);
    // the token leaves its cell: one customer, and one table if it is a head
    const int32_t dv = 1 + (r0 << kCountBits);

    // Stirling ratio pairs of every cell, the own cell without the token
    float2 qv[KPL];
    int32_t own_nt = 0;
#pragma unroll
    for (int j = 0; j < KPL; ++j) {
        const bool own = (kbase + j == k0);
        own_nt = own ? cur.n[j] : own_nt;
        const uint32_t v = (uint32_t)(cur.n[j] - (own ? dv : 0));
        const uint32_t cn = v & kCountMax, ct = v >> kCountBits;
        uint32_t ix = ((cn * (cn + 1)) >> 1) + ct;
        ix = ix < q_last ? ix : q_last;
        // 32-bit byte offsets while the ratio table is below 4 GiB (2^29 pairs),
        // else 64-bit addresses
        if constexpr (BIGQ)
            qv[j] = A.Q[ix];
        else
            qv[j] = *reinterpret_cast<const float2 *>(reinterpret_cast<const char *>(A.Q) +
                                                      (ix << 3));
    }
    // removed-customer constants of the own topic (a small table that stays
    // in cache), requested with the gathers; their addresses are wave-uniform,
    // so each is one load from a scalar base address, with no per-lane 64-bit
    // address arithmetic
    const float f0k = A.fk[W.gK + k0];
    const float f1k = A.fk[(int64_t)(1 + r0) * A.GK + W.gK + k0];
    // rows of token i + 2 (past the end: the last token's rows again,
    // unused), requested after the gathers so that waiting for the gathers
    // does not wait for them
    asm volatile("" ::: "memory");
    load_rows<KPL>(A, W, x + 2, fill);
    __builtin_amdgcn_s_setprio(0);
    // only head of a cell that keeps other customers: point mass
    const int32_t nt0 = readlane(own_nt, k0 / KPL);
    const bool sole = r0 && (nt0 >> kCountBits) == 1 && (nt0 & kCountMax) > 1;

    int32_t result = zr0;
    float u = -1.0f;
    if (!sole) {
        const float doc0 = A.alpha + (float)(W.c_lds[k0] - 1);
        const float m1k0 = doc0 * f1k, m0k0 = doc0 * f0k;

        // Shadow-base counts of the token's word: the 16-bit copy, whose
        // cells are exact in the 16-bit launch.  In the 32-bit launch (some
        // count above 65535) a token whose row saturates a cell in any lane
        // reads the lanes' slices of B itself (a rare, wave-uniform branch
        // whose load waits for the loads in flight).
        int32_t bv[KPL];
#pragma unroll
        for (int j = 0; j < KPL; ++j) bv[j] = cur.b(j);
        if constexpr (WIDE) {
            bool sat = false;
#pragma unroll
            for (int j = 0; j < KPL; ++j) sat = sat || (bv[j] == 0xFFFF);
            if (__ballot(sat)) {
                const int64_t wrow = (int64_t)(readlane(W.gw_c, x) - W.gV) * A.Kp;
                load_row<KPL>(bv, A.B + wrow, kbase, A.Kp);
            }
        }

        // weights and lane-local inclusive prefix sums
        float a0[KPL], a1[KPL];
        lds_row<KPL>(a0, W.a0_lds, lane);
        lds_row<KPL>(a1, W.a1_lds, lane);
        float s[NO];
        float acc = 0.0f;
#pragma unroll
        for (int j = 0; j < KPL; ++j) {
            const bool own = (kbase + j == k0);
            const float bw = A.gamma + (float)(bv[j] - (own ? r0 : 0));
            const float m1 = own ? m1k0 : a1[j];
            const float m0 = own ? m0k0 : a0[j];
            const float w1 = m1 * bw * qv[j].y;
            const float w0 = m0 * qv[j].x;
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
        __builtin_amdgcn_s_setprio(3);
        const float incl = wave_inclusive_sum(acc);
        const float excl = wave_shift_right(incl);
        const float total = readlane_f(incl, 63);

        u = readlane_f(W.u_c, x);
        const float target = u * total;

        // prefixes are monotone, so the number of this lane's prefixes at or
        // below the target is the index of its first crossing
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
            // the two prefixes around the crossing; re-decide in fp64 if the
            // target is within rounding distance of either
            const float hi = readlane_f(excl + s[cL], L);
            const float lo = readlane_f(cL > 0 ? excl + s[cL > 0 ? cL - 1 : 0] : excl, L);
            const float margin = fix_margin<KPL>() * total;
            fix = (target - lo < margin) || (hi - target < margin);
            jstar = L * NO + cL;
        }
        if (fix) {
            // The draw is within rounding distance of a CDF boundary (or the
            // fp32 scan found no crossing): take it again with fp64 weights
            // from the integer counts, fp64 prefix sums and the same uniform.
            // Rolled loops keep this rare path from raising the kernel's
            // register count; each step picks its cell's counts out of the
            // rows in registers, so its loads (the group's totals and the
            // cell's fp64 ratio pair) go out together: one memory round trip.
            const ExactCtx &X = *A.exact;
            const int32_t *__restrict__ Ng = X.Ngk + W.gK;
            const int32_t *__restrict__ Tg = X.Tgk + W.gK;
            double acc64 = 0.0;
            int32_t last64 = -1;
#pragma unroll 1
            for (int j = 0; j < KPL; ++j) {
                const int32_t k = kbase + j;
                if (k >= A.K) break;
                const Exact e =
                    exact_pair(X, k, k0, r0, pick(cur.n, j),
                                         exact_b<KPL, WIDE>(A, W, x, cur, j), W.c_lds[k], Ng, Tg);
                acc64 += e.w1;
                if (e.w1 > 0.0) last64 = 2 * j;
                acc64 += e.w0;
                if (e.w0 > 0.0) last64 = 2 * j + 1;
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
            // the first outcome whose prefix exceeds the target: only lanes
            // whose prefix ends above the target walk, each up to its first
            int32_t cand64 = -1;
            if (incl64 > target64) {
#pragma unroll 1
                for (int j = 0; j < KPL; ++j) {
                    const int32_t k = kbase + j;
                    if (k >= A.K) break;
                    const Exact e = exact_pair(X, k, k0, r0, pick(cur.n, j),
                                               exact_b<KPL, WIDE>(A, W, x, cur, j),
                                               W.c_lds[k], Ng, Tg);
                    run += e.w1;
                    if (e.w1 > 0.0 && run > target64) {
                        cand64 = 2 * j;
                        break;
                    }
                    run += e.w0;
                    if (e.w0 > 0.0 && run > target64) {
                        cand64 = 2 * j + 1;
                        break;
                    }
                }
            }
            // (the last positive outcome if rounding leaves none)
            jstar = -1;
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
        __builtin_amdgcn_s_setprio(0);
        if (jstar >= 0) {
            const int32_t k1 = jstar >> 1, r1 = 1 - (jstar & 1);
            result = zr_pack(k1, r1);
            // DS operations of one wave execute in order, so the next token's
            // reads of the LDS rows see this update
            if (lane == 0 && k1 != k0) {
                const int32_t ca = W.c_lds[k0] - 1, cb = W.c_lds[k1] + 1;
                W.c_lds[k0] = ca;
                W.c_lds[k1] = cb;
                const float da = A.alpha + (float)ca, db = A.alpha + (float)cb;
                W.a0_lds[lds_pos<KPL>(k0)] = da * W.f0_lds[k0];
                W.a1_lds[lds_pos<KPL>(k0)] = da * W.f1_lds[k0];
                W.a0_lds[lds_pos<KPL>(k1)] = db * W.f0_lds[k1];
                W.a1_lds[lds_pos<KPL>(k1)] = db * W.f1_lds[k1];
            }
        }
    }
    if constexpr (TRACE) {
        if (lane == 0 && i >= A.tr_begin && i < A.tr_end) A.tr_u[i - A.tr_begin] = u;
    }
    if (lane == x) W.out_c = result;
}

// One document on the calling wavefront; the LDS arrays are the workgroup's
// (the live document row c[k], the group's per-topic constants f0, f1 and the
// products a0 = (alpha + c) f0, a1 = (alpha + c) f1, kept in step with c;
// interleaved layout).
template <int KPL, bool TRACE, bool WIDE, bool BIGQ>
__device__ __forceinline__ void sample_doc(const SampleArgs &A, int32_t d, int32_t *c_lds,
                                           float *f0_lds, float *f1_lds, float *a0_lds,
                                           float *a1_lds)
{
    DocWave<KPL> W;
    const int64_t beg = A.doc_off[d];
    W.end = A.doc_off[d + 1];
    if (beg >= W.end) return;
    W.lane = threadIdx.x;
    const int32_t g = A.doc_group[d];
    W.kbase = W.lane * KPL;
    W.gV = g * A.V;
    W.gK = (int64_t)g * A.Kp;
    W.c_lds = c_lds;
    W.f0_lds = f0_lds;
    W.f1_lds = f1_lds;
    W.a0_lds = a0_lds;
    W.a1_lds = a1_lds;
    const int32_t lane = W.lane, kbase = W.kbase;
    const int64_t end = W.end, last = end - 1;

    {
        float f0[KPL], f1[KPL];
        load_slice_f<KPL>(f0, A.f0 + W.gK, kbase, A.Kp);
        load_slice_f<KPL>(f1, A.f1 + W.gK, kbase, A.Kp);
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
        const int32_t k = kbase + j;
        const float doc = A.alpha + (float)c_lds[k];
        a0_lds[lds_pos<KPL>(k)] = doc * f0_lds[k];
        a1_lds[lds_pos<KPL>(k)] = doc * f1_lds[k];
    }
    __syncthreads();

    W.cb = beg;
    W.out_c = 0;
    load_stream<KPL>(A, W, last);

    // three row buffers: the current token's and the next two tokens'
    Rows<KPL> ra, rb, rc;
    load_rows<KPL>(A, W, 0, ra);
    load_rows<KPL>(A, W, 1, rb);
    int32_t x = 0;  // position of token i in the stream registers
    for (int64_t i = beg; i < end; i += 3, x += 3) {
        if (x == kChunk) {
            if (lane < kChunk) A.zr_new[W.cb + lane] = W.out_c;
            W.cb += kChunk;
            x = 0;
            load_stream<KPL>(A, W, last);
        }
        sample_token<KPL, TRACE, WIDE, BIGQ>(A, W, x, ra, rc);
        if (i + 1 < end) sample_token<KPL, TRACE, WIDE, BIGQ>(A, W, x + 1, rb, ra);
        if (i + 2 < end) sample_token<KPL, TRACE, WIDE, BIGQ>(A, W, x + 2, rc, rb);
    }
    if (lane < end - W.cb) A.zr_new[W.cb + lane] = W.out_c;
}

// Launched twice per sweep, once per width of the shadow-base rows; the
// launch that does not match the flag set by the count rebuild returns.  The
// 16-bit width (the common case) takes one workgroup per document; blocks are
// dealt round-robin over the 8 XCDs, and each XCD gets a contiguous range of
// documents so a group's hot rows stay in its L2.  The 32-bit width runs as a
// persistent grid whose workgroups claim the documents of their XCD's range
// one at a time, so that its launch costs almost nothing when it returns.
template <int KPL, bool TRACE, bool WIDE, bool BIGQ>
__global__ void __launch_bounds__(64, (KPL <= 8 ? 4 : 2)) k_sample(SampleArgs A)
{
    __shared__ int32_t c_lds[64 * KPL];
    __shared__ float f0_lds[64 * KPL];
    __shared__ float f1_lds[64 * KPL];
    __shared__ __attribute__((aligned(16))) float a0_lds[64 * KPL];
    __shared__ __attribute__((aligned(16))) float a1_lds[64 * KPL];

    if ((*A.wide != 0) != WIDE) return;
    if constexpr (!WIDE) {
        const int32_t b = blockIdx.x;
        const int32_t d = (b & 7) * A.docs_per_xcd + (b >> 3);
        if (d >= A.D) return;
        sample_doc<KPL, TRACE, WIDE, BIGQ>(A, d, c_lds, f0_lds, f1_lds, a0_lds, a1_lds);
    } else {
        const int32_t xcd = blockIdx.x & 7;
        for (;;) {
            int32_t i = 0;
            if (threadIdx.x == 0) i = atomicAdd(&A.claim[xcd], 1);
            i = __shfl(i, 0);
            if (i >= A.docs_per_xcd) break;
            const int32_t d = xcd * A.docs_per_xcd + i;
            if (d >= A.D) break;
            sample_doc<KPL, TRACE, WIDE, BIGQ>(A, d, c_lds, f0_lds, f1_lds, a0_lds, a1_lds);
        }
        // the last workgroup to finish clears the claims for the next launch
        if (threadIdx.x == 0) {
            __threadfence();
            if (atomicAdd(&A.claim[8], 1) == (int32_t)gridDim.x - 1) {
#pragma unroll 1
                for (int u = 0; u < 9; ++u) A.claim[u] = 0;
            }
        }
    }
}

// workgroups of the persistent launch: a wavefront slot each on 256 compute
// units at 4 wavefronts per SIMD (fewer when the documents are fewer)
constexpr int32_t kPersistentBlocks = 4096;

template <int KPL, bool BIGQ>
hipError_t launch_kpl_q(const SampleArgs &A, bool trace, hipStream_t st)
{
    const unsigned grid = (unsigned)(8 * A.docs_per_xcd);
    const unsigned pgrid = grid < (unsigned)kPersistentBlocks ? grid : (unsigned)kPersistentBlocks;
    if (trace) {
        hipLaunchKernelGGL((k_sample<KPL, true, false, BIGQ>), dim3(grid), dim3(64), 0, st, A);
        hipLaunchKernelGGL((k_sample<KPL, true, true, BIGQ>), dim3(pgrid), dim3(64), 0, st, A);
    } else {
        hipLaunchKernelGGL((k_sample<KPL, false, false, BIGQ>), dim3(grid), dim3(64), 0, st, A);
        hipLaunchKernelGGL((k_sample<KPL, false, true, BIGQ>), dim3(pgrid), dim3(64), 0, st, A);
    }
    return hipGetLastError();
}

template <int KPL>
hipError_t launch_kpl(const SampleArgs &A, bool trace, hipStream_t st)
{
    return A.nQ > kSmallQ ? launch_kpl_q<KPL, true>(A, trace, st)
                          : launch_kpl_q<KPL, false>(A, trace, st);
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

// Rows are padded to whole 128-byte lines of int32 cells (so a row read
// touches no partial line); 64 KPL >= Kp always holds.
int32_t padded_K(int32_t K) { return (K + 31) / 32 * 32; }

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
    A.nt16 = b.nt16;
    A.tok_narrow = b.tok_narrow;
    A.B = b.B;
    A.B16 = b.B16;
    A.wide = b.wide;
    A.claim = b.claim;
    A.f0 = b.f0;
    A.f1 = b.f1;
    A.fk = b.fk;
    A.Q = b.Q;
    A.exact = b.exact;
    A.tr_w = tr_w;
    A.tr_u = tr_u;
    A.tr_begin = tr_begin;
    A.tr_end = tr_end;
    A.seed = seed;
    A.D = m.D;
    A.V = m.V;
    A.K = m.K;
    A.Kp = m.Kp;
    A.nQ = tri_index(m.ncap, 0);
    A.GK = (int64_t)m.G * m.Kp;
    A.docs_per_xcd = (m.D + 7) / 8;
    A.sweep = sweep;
    A.alpha = (float)m.alpha;
    A.gamma = (float)m.gamma;
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
