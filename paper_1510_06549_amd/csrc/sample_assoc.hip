// sample_assoc.hip -- the per-sweep resampling kernel of the model with word
// associations (non-identity transformation matrices P^g), gfx950 wave64.
//
// In the full SPDP model a new table of topic k in group g first takes a
// source word v from the shadow base phi0_k and then serves word w with
// probability p_{g,w,v} (column v of P^g is a distribution over words).  Each
// table head carries its source, stored as its slot s in the source list of
// its (g, w) row, and the shadow-base table counts B[v][k] are keyed by
// source.  A token has K (S + 1) outcomes: for each topic k the head outcomes
// (k, r = 1, slot s), s = 0 .. S - 1, then (k, r = 0), with the weights of
// Eq. SPDP-sampling-w-z-r1 (with p_{i,w,v} and the source-keyed base count)
// and Eq. SPDP-sampling-w-z-r0:
//   W(k, 1, s) = p_s (alpha + c'_k) f1[g][k] (gamma + B'[v_s][k]) Q1(n', t')
//   W(k, 0)    = (alpha + c'_k) f0[g][k] Q0(n', t')
// where the token's own customer, table and source count are removed (the
// removed-customer constants of its topic come from fk, as in the plain
// kernel).  Slots past the end of a shorter list have p = 0.  The only head of
// a cell that keeps other customers must stay that cell's head (every other
// topic or r has joint probability zero), but its source is free: then only
// its own topic's head slots carry weight, W(k0, 1, s) = p_s (gamma + B'[v_s][k0]).
//
// Layout and scheduling follow the plain kernel: one wavefront per document,
// the shared counts from the sweep-start snapshot, the document's row c[k]
// live in LDS.  Lane l owns KPL contiguous topics; per token the wave loads
// the packed count row of (g, w) and the SP 16-bit (or 32-bit) shadow-base
// rows of the row's sources, one token ahead of use (two register sets
// alternate).  The token stream (row index, state, uniform and the row's
// source record) is read 64 tokens at a time, one token per lane.
//
// The draw: per lane, the running prefix at the end of each of its topics
// (head slots first, as one factored term p-weighted over the sources, then
// r = 0); a DPP wave scan gives each lane's offset; the crossing topic is the
// first whose prefix exceeds u * total, and its slot prefixes are formed again
// in the crossing lane with the same roundings.  A target within fp32 rounding
// distance of a boundary is decided again with fp64 weights from the integer
// counts, as in the plain kernel.
#include "sampler_common.hpp"

namespace spdp {

namespace {

struct AssocArgs {
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
    const int32_t *srcrec;  // [G V][2 SP]: sources, then p (fp32 bits)
    const ExactCtx *exact;
    float *tr_w;
    float *tr_u;
    int64_t tr_begin, tr_end;
    uint64_t seed;
    int32_t D, V, K, Kp, S;  // S: longest source list (outcomes per topic S + 1)
    int64_t nQ, GK;
    int32_t docs_per_xcd;
    uint32_t sweep;
    float alpha, gamma;
};

// Tokens per step of the token stream (a multiple of the two alternating row
// sets; the one-ahead look-up stays inside the 64 stream registers).
constexpr int32_t kAChunk = 48;

// The rows one token needs: this lane's slice of its packed count row and of
// the shadow-base rows of its SP sources.
template <int KPL, int SP, bool WIDE>
struct ARows {
    static constexpr int NB = WIDE ? KPL : (KPL + 1) / 2;
    int32_t n[KPL];
    uint32_t bw[SP][NB];
    __device__ __forceinline__ int32_t b(int s, int j) const
    {
        if constexpr (WIDE) return (int32_t)bw[s][j];
        else return (int32_t)((bw[s][j >> 1] >> (16 * (j & 1))) & 0xFFFFu);
    }
    // the same for a wave-uniform j that is not a compile-time constant
    __device__ __forceinline__ int32_t b_at(int s, int j) const
    {
        if constexpr (WIDE) return (int32_t)pick(bw[s], j);
        else return (int32_t)((pick(bw[s], j >> 1) >> (16 * (j & 1))) & 0xFFFFu);
    }
};

template <int KPL, int SP>
struct AWave {
    int32_t lane, kbase, gV;
    int64_t gK, cb, end;
    int32_t *c_lds;
    float *f0_lds, *f1_lds, *a0_lds, *a1_lds;
    // token stream: lane l holds token cb + l (lanes past the document's end
    // repeat its last token): row index, packed state, narrow-row flag,
    // uniform, and the source record of its row
    int32_t gw_c, zr_c, nar_c, out_c;
    float u_c;
    int32_t src_c[SP];
    float p_c[SP];
};

// lds_row with each 16-byte chunk pinned as one value, so that the compiler
// keeps whole-chunk reads (split 4-byte reads at a 16-byte lane stride would
// conflict on the LDS banks)
template <int KPL>
__device__ __forceinline__ void lds_row_whole(float (&v)[KPL], const float *base, int32_t lane)
{
    if constexpr (KPL % 4 == 0) {
#pragma unroll
        for (int c = 0; c < KPL / 4; ++c) {
            typedef float f4 __attribute__((ext_vector_type(4)));
            f4 x = reinterpret_cast<const f4 *>(base)[c * 64 + lane];
            asm volatile("" : "+v"(x));
            v[4 * c + 0] = x[0];
            v[4 * c + 1] = x[1];
            v[4 * c + 2] = x[2];
            v[4 * c + 3] = x[3];
        }
    } else {
        lds_row<KPL>(v, base, lane);
    }
}

// Distance from a CDF boundary, as a fraction of the total, below which the
// fp32 decision is taken again in fp64.  To first order in u = 2^-24, as in
// the plain kernel: a topic's head term carries at most 10 + SP relative
// roundings (the factor (alpha + c) f1 Q1 six, each source's p and gamma + B
// three, the fused p-weighted sum SP, the product one) and its r = 0 term 6;
// the summations of a boundary and of the total behind the target each add
// at most (2 KPL + 5)u; the target, its lane offset, the compared boundary
// and the distance one rounding each; the crossing topic's slot prefixes are
// formed with the same roundings.  So the fp32 distance is within
// (4 KPL + SP + 24)u of the exact one, and outside (4 KPL + SP + 32)u both
// decisions agree.
template <int KPL, int SP>
__device__ __forceinline__ float fix_margin()
{
    return (float)(4 * KPL + SP + 32) * 5.97e-8f;
}

template <int KPL, int SP, bool WIDE>
__device__ __forceinline__ void load_arows(const AssocArgs &A, const AWave<KPL, SP> &W, int32_t x,
                                           ARows<KPL, SP, WIDE> &R)
{
    const int32_t q = readlane(W.gw_c, x);
    // a narrow row as its 16-bit copy (half the bytes), widened at use
    load_count_row<KPL>(R.n, A.nt, A.nt16, q, W.kbase, A.Kp, readlane(W.nar_c, x) != 0);
#pragma unroll
    for (int s = 0; s < SP; ++s) {
        const int64_t vrow = (int64_t)readlane(W.src_c[s], x) * A.Kp;
        if constexpr (WIDE)
            load_row<KPL>(reinterpret_cast<int32_t(&)[KPL]>(R.bw[s]), A.B + vrow, W.kbase, A.Kp);
        else
            load_half_row<KPL>(R.bw[s], A.B16 + vrow, W.kbase, A.Kp);
    }
}

template <int KPL, int SP>
__device__ __forceinline__ void load_astream(const AssocArgs &A, AWave<KPL, SP> &W, int64_t last)
{
    const int64_t t = min(W.cb + W.lane, last);
    W.gw_c = A.gw[t];
    W.zr_c = A.zr_old[t];
    W.nar_c = A.tok_narrow[t];
    const int32_t *rec = A.srcrec + (int64_t)W.gw_c * (2 * SP);
    if constexpr (SP == 1) {
        const int2 x = *reinterpret_cast<const int2 *>(rec);
        W.src_c[0] = x.x;
        W.p_c[0] = __int_as_float(x.y);
    } else {
        int32_t v[2 * SP];
#pragma unroll
        for (int c = 0; c < SP / 2; ++c) {
            const int4 x = reinterpret_cast<const int4 *>(rec)[c];
            v[4 * c + 0] = x.x;
            v[4 * c + 1] = x.y;
            v[4 * c + 2] = x.z;
            v[4 * c + 3] = x.w;
        }
#pragma unroll
        for (int s = 0; s < SP; ++s) {
            W.src_c[s] = v[s];
            W.p_c[s] = __int_as_float(v[SP + s]);
        }
    }
    const uint32_t xr = philox_x0(A.seed, (uint64_t)(W.cb + W.lane), A.sweep, kPurposeSample);
    W.u_c = (float)(xr >> 8) * (1.0f / 16777216.0f);
#pragma unroll
    for (int s = 0; s < SP; ++s) asm volatile("" ::"v"(W.src_c[s]), "v"(W.p_c[s]));
    asm volatile("" ::"v"(W.gw_c), "v"(W.zr_c), "v"(W.nar_c));
}

// fp64 weights of topic k's SP + 1 outcomes from the integer counts (the
// packed cell nt_raw, the source-keyed base counts b_raw of the row's
// sources, the document count c_raw), the fp64 ratio pairs and the fp64 p of
// the row (the rare boundary path).
template <int SP>
__device__ void exact_topic(const ExactCtx &X, int32_t k, int32_t k0, int32_t r0, int32_t s0,
                            bool sole, int32_t nt_raw, const int32_t (&b_raw)[SP], int32_t c_raw,
                            const int32_t *Ng, const int32_t *Tg, const double *p64,
                            double (&w1)[SP], double &w0)
{
    const int32_t del = (k == k0) ? 1 : 0;
    w0 = 0.0;
    if (sole) {
#pragma unroll
        for (int s = 0; s < SP; ++s) {
            const int32_t bv = b_raw[s] - ((del && s == s0) ? 1 : 0);
            w1[s] = del ? p64[s] * (X.gamma + (double)bv) : 0.0;
        }
        return;
    }
    const int32_t n_raw = nt_raw & kCountMax, t_raw = nt_raw >> kCountBits;
    const int64_t nn = n_raw - del, tt = t_raw - del * r0;
    const double N = (double)(Ng[k] - del), T = (double)(Tg[k] - del * r0);
    const double Bt = (double)(X.Bk[k] - del * r0);
    const double doc = X.alpha + (double)(c_raw - del);
    const double2 qq = X.Q64[exact_q_index(X, (int32_t)nn, (int32_t)tt)];
    const double q0 = qq.x, q1 = qq.y;
#pragma unroll
    for (int s = 0; s < SP; ++s) {
        const int32_t bv = b_raw[s] - ((del && r0 && s == s0) ? 1 : 0);
        w1[s] = p64[s] * doc * (X.b + X.a * T) / (X.b + N) * (X.gamma + (double)bv) /
                (X.Vgamma + Bt) * q1;
    }
    w0 = doc / (X.b + N) * q0;
}

// Token cb + x: sample it with the rows in `cur` and request the rows of the
// next token into `fill`.
template <int KPL, int SP, bool WIDE, bool BIGQ>
__device__ __forceinline__ void sample_token_assoc(const AssocArgs &A, AWave<KPL, SP> &W,
                                                   int32_t x, ARows<KPL, SP, WIDE> &cur,
                                                   ARows<KPL, SP, WIDE> &fill)
{
    const int32_t lane = W.lane, kbase = W.kbase;
    const int64_t i = W.cb + x;
    if (readlane(W.nar_c, x)) widen_cells<KPL>(cur.n, kbase);

    const int32_t zr0 = readlane(W.zr_c, x);
    const int32_t k0 = zr_topic(zr0), r0 = zr0 & 1, s0 = zr_slot(zr0);
    const uint32_t q_last = (uint32_t)(A.nQ - 1);
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
    asm volatile("" ::: "memory");
    load_arows<KPL, SP, WIDE>(A, W, x + 1, fill);

    const int32_t nt0 = readlane(own_nt, k0 / KPL);
    const bool sole = r0 && (nt0 >> kCountBits) == 1 && (nt0 & kCountMax) > 1;

    float p[SP];
#pragma unroll
    for (int s = 0; s < SP; ++s) p[s] = readlane_f(W.p_c[s], x);

    const float doc0 = A.alpha + (float)(W.c_lds[k0] - 1);
    const float m1k0 = doc0 * f1k, m0k0 = doc0 * f0k;
    float a0[KPL], a1[KPL];
    lds_row_whole<KPL>(a0, W.a0_lds, lane);
    lds_row_whole<KPL>(a1, W.a1_lds, lane);

    // per topic: the base weight of each source slot, their p-weighted sum,
    // the factor of the head outcomes and the running prefix at the topic end
    // (branch-free: the sole-head case is a uniform select, so the compiler
    // keeps the LDS rows as whole 16-byte reads)
    float hq[KPL], e[KPL];
    float acc = 0.0f;
#pragma unroll
    for (int j = 0; j < KPL; ++j) {
        const bool own = (kbase + j == k0);
        float beta = 0.0f;
#pragma unroll
        for (int s = 0; s < SP; ++s) {
            const float bv = A.gamma + (float)(cur.b(s, j) - ((own && r0 && s == s0) ? 1 : 0));
            beta = __fmaf_rn(p[s], bv, beta);
        }
        const float h_draw = __fmul_rn(own ? m1k0 : a1[j], qv[j].y);
        const float w0_draw = __fmul_rn(own ? m0k0 : a0[j], qv[j].x);
        hq[j] = sole ? (own ? 1.0f : 0.0f) : h_draw;
        const float w0 = sole ? 0.0f : w0_draw;
        acc = __fadd_rn(acc, __fmul_rn(hq[j], beta));
        acc = __fadd_rn(acc, w0);
        e[j] = acc;
    }
    if (A.tr_w != nullptr && i >= A.tr_begin && i < A.tr_end) {
        // debug trace: every outcome's weight, formed again from the same values
#pragma unroll
        for (int j = 0; j < KPL; ++j) {
            if (kbase + j >= A.K) continue;
            const bool own = (kbase + j == k0);
            float *o = A.tr_w + (i - A.tr_begin) * (int64_t)A.K * (A.S + 1) +
                       (int64_t)(kbase + j) * (A.S + 1);
#pragma unroll
            for (int s = 0; s < SP; ++s) {
                if (s < A.S) {
                    const float bv =
                        A.gamma + (float)(cur.b(s, j) - ((own && r0 && s == s0) ? 1 : 0));
                    o[s] = hq[j] * (p[s] * bv);
                }
            }
            o[A.S] = sole ? 0.0f : __fmul_rn(own ? m0k0 : a0[j], qv[j].x);
        }
    }
    // the serial scan and draw at wave priority 3, above the weight loops of
    // the other wavefronts on the SIMD, so that the draw resolves without
    // queueing behind their vector work
    __builtin_amdgcn_s_setprio(3);
    const float incl = wave_inclusive_sum(acc);
    const float excl = wave_shift_right(incl);
    const float total = readlane_f(incl, 63);
    const float u = readlane_f(W.u_c, x);
    const float target = u * total;
    const float rel = target - excl;
    int32_t cnt = 0;
#pragma unroll
    for (int j = 0; j < KPL; ++j) cnt += (e[j] <= rel) ? 1 : 0;
    const unsigned long long cross = __ballot(cnt < KPL);

    int32_t k1 = k0, r1 = r0, s1 = s0;
    bool fix = true;
    if (cross) {
        const int32_t L = __ffsll((long long)cross) - 1;
        const int32_t jc = readlane(cnt, L);
        // topic jc of every lane (only lane L's is used): its prefix before,
        // its head factor and its slot base weights, with the same roundings
        float before = 0.0f, hsel = 0.0f, esel = 0.0f;
        float bsel[SP];
#pragma unroll
        for (int s = 0; s < SP; ++s) bsel[s] = 0.0f;
#pragma unroll
        for (int j = 0; j < KPL; ++j) {
            if (j == jc) {
                const bool own = (kbase + j == k0);
                before = (j > 0) ? e[j > 0 ? j - 1 : 0] : 0.0f;
                hsel = hq[j];
                esel = e[j];
#pragma unroll
                for (int s = 0; s < SP; ++s)
                    bsel[s] = A.gamma + (float)(cur.b(s, j) - ((own && r0 && s == s0) ? 1 : 0));
            }
        }
        // slot prefixes: before + hq * (running p-weighted sum), the last of
        // them equal to the head part of the stage above
        int32_t slot = SP;  // SP: the r = 0 outcome
        float lo = 0.0f, hi = 0.0f, prev = before, bp = 0.0f;
        bool found = false;
#pragma unroll
        for (int s = 0; s < SP; ++s) {
            bp = __fmaf_rn(p[s], bsel[s], bp);
            const float pre = __fadd_rn(before, __fmul_rn(hsel, bp));
            if (!found && pre > rel) {
                found = true;
                slot = s;
                lo = prev;
                hi = pre;
            }
            prev = pre;
        }
        if (!found) {
            lo = prev;
            hi = esel;
        }
        const int32_t slotL = readlane(slot, L);
        const float loL = readlane_f(lo, L), hiL = readlane_f(hi, L);
        const float relL = readlane_f(rel, L);
        const float margin = fix_margin<KPL, SP>() * total;
        // the crossing must lie inside this topic (hi > rel >= lo), else the
        // fp32 prefixes disagree and the draw is decided in fp64
        fix = !(hiL > relL) || (relL - loL < margin) || (hiL - relL < margin);
        k1 = L * KPL + jc;
        r1 = slotL < SP ? 1 : 0;
        s1 = slotL < SP ? slotL : 0;
    }
    if (fix) {
        // fp64 weights from the integer counts, fp64 prefix sums, the same
        // uniform.  Rolled loops keep this rare path from raising the register
        // count; each step picks its cell's counts out of the rows in
        // registers, so its loads (the group's totals and the cell's fp64
        // ratio pair) go out together: one memory round trip.
        const int32_t q = readlane(W.gw_c, x);
        const ExactCtx &X = *A.exact;
        const int32_t *__restrict__ Ng = X.Ngk + W.gK;
        const int32_t *__restrict__ Tg = X.Tgk + W.gK;
        const double *__restrict__ p64 = X.p64 + (int64_t)q * SP;
        double acc64 = 0.0;
        int32_t lastp = -1;
#pragma unroll 1
        for (int j = 0; j < KPL; ++j) {
            const int32_t k = kbase + j;
            if (k >= A.K) break;
            int32_t bj[SP];
#pragma unroll
            for (int s = 0; s < SP; ++s) bj[s] = cur.b_at(s, j);
            double w1[SP], w0;
            exact_topic<SP>(X, k, k0, r0, s0, sole, pick(cur.n, j), bj, W.c_lds[k], Ng, Tg, p64,
                            w1, w0);
#pragma unroll
            for (int s = 0; s < SP; ++s) {
                acc64 += w1[s];
                if (w1[s] > 0.0) lastp = j * (SP + 1) + s;
            }
            acc64 += w0;
            if (w0 > 0.0) lastp = j * (SP + 1) + SP;
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
        // the first outcome whose prefix exceeds the target: only lanes whose
        // prefix ends above the target walk, each up to its first
        int32_t cand = -1;
        if (incl64 > target64) {
#pragma unroll 1
            for (int j = 0; j < KPL; ++j) {
                const int32_t k = kbase + j;
                if (k >= A.K) break;
                int32_t bj[SP];
#pragma unroll
                for (int s = 0; s < SP; ++s) bj[s] = cur.b_at(s, j);
                double w1[SP], w0;
                exact_topic<SP>(X, k, k0, r0, s0, sole, pick(cur.n, j), bj, W.c_lds[k], Ng, Tg,
                                p64, w1, w0);
#pragma unroll
                for (int s = 0; s < SP; ++s) {
                    run += w1[s];
                    if (cand < 0 && w1[s] > 0.0 && run > target64) cand = j * (SP + 1) + s;
                }
                run += w0;
                if (cand < 0 && w0 > 0.0 && run > target64) cand = j * (SP + 1) + SP;
                if (cand >= 0) break;
            }
        }
        // (the last positive outcome if rounding leaves none)
        int32_t jl = -1, Lx = -1;
        const unsigned long long m2 = __ballot(cand >= 0);
        if (m2) {
            Lx = __ffsll((long long)m2) - 1;
            jl = readlane(cand, Lx);
        } else {
            const unsigned long long m3 = __ballot(lastp >= 0);
            if (m3) {
                Lx = 63 - __clzll((long long)m3);
                jl = readlane(lastp, Lx);
            }
        }
        if (jl >= 0) {
            const int32_t sl = jl % (SP + 1);
            k1 = Lx * KPL + jl / (SP + 1);
            r1 = sl < SP ? 1 : 0;
            s1 = sl < SP ? sl : 0;
        } else {
            k1 = k0;
            r1 = r0;
            s1 = s0;
        }
    }
    __builtin_amdgcn_s_setprio(0);
    // DS operations of one wave execute in order, so the next token's reads of
    // the LDS rows see this update
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
    if (A.tr_u != nullptr && lane == 0 && i >= A.tr_begin && i < A.tr_end)
        A.tr_u[i - A.tr_begin] = u;
    if (lane == x) W.out_c = zr_pack(k1, r1, s1);
}

// Waves per SIMD the kernel is built for: the LDS rows (20 B per topic slot,
// 160 KiB per CU) and an estimate of the registers (two row sets, the per-topic
// values of the draw, and about 90 for the rest, fitted to the compiler's
// allocation) bound it, at most 4.
template <int KPL, int SP, bool WIDE>
constexpr int assoc_waves()
{
    constexpr int set = KPL + SP * ARows<KPL, SP, WIDE>::NB;
    constexpr int regs = 2 * set + 3 * KPL + 2 * SP + 90;
    constexpr int by_lds = (160 * 1024) / (20 * 64 * KPL) / 4;
    constexpr int by_regs = 512 / regs;
    constexpr int w = by_lds < by_regs ? by_lds : by_regs;
    return w > 4 ? 4 : (w < 1 ? 1 : w);
}

// One document on the calling wavefront, with the workgroup's LDS arrays (as
// in the plain sampler).
template <int KPL, int SP, bool WIDE, bool BIGQ>
__device__ __forceinline__ void sample_doc_assoc(const AssocArgs &A, int32_t d, int32_t *c_lds,
                                                 float *f0_lds, float *f1_lds, float *a0_lds,
                                                 float *a1_lds)
{
    AWave<KPL, SP> W;
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
    for (int64_t i = beg + lane; i < end; i += 64) atomicAdd(&c_lds[zr_topic(A.zr_old[i])], 1);
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
    load_astream<KPL, SP>(A, W, last);
    ARows<KPL, SP, WIDE> ra, rb;
    load_arows<KPL, SP, WIDE>(A, W, 0, ra);
    int32_t x = 0;
    for (int64_t i = beg; i < end; i += 2, x += 2) {
        if (x == kAChunk) {
            if (lane < kAChunk) A.zr_new[W.cb + lane] = W.out_c;
            W.cb += kAChunk;
            x = 0;
            load_astream<KPL, SP>(A, W, last);
        }
        sample_token_assoc<KPL, SP, WIDE, BIGQ>(A, W, x, ra, rb);
        if (i + 1 < end) sample_token_assoc<KPL, SP, WIDE, BIGQ>(A, W, x + 1, rb, ra);
    }
    if (lane < end - W.cb) A.zr_new[W.cb + lane] = W.out_c;
}

// Launched twice per sweep, once per width of the shadow-base rows; the
// launch that does not match the flag set by the rebuild returns.  As in the
// plain sampler, the 16-bit width takes one workgroup per document (each XCD
// a contiguous range) and the 32-bit width runs as a persistent grid whose
// workgroups claim their XCD's documents one at a time.
template <int KPL, int SP, bool WIDE, bool BIGQ>
__global__ void __launch_bounds__(64, (assoc_waves<KPL, SP, WIDE>())) k_sample_assoc(AssocArgs A)
{
    __shared__ int32_t c_lds[64 * KPL];
    __shared__ float f0_lds[64 * KPL];
    __shared__ float f1_lds[64 * KPL];
    __shared__ __attribute__((aligned(16))) float a0_lds[64 * KPL];
    __shared__ __attribute__((aligned(16))) float a1_lds[64 * KPL];

    if ((*A.wide != 0) != WIDE) return;
    if constexpr (!WIDE) {
        const int32_t bidx = blockIdx.x;
        const int32_t d = (bidx & 7) * A.docs_per_xcd + (bidx >> 3);
        if (d >= A.D) return;
        sample_doc_assoc<KPL, SP, WIDE, BIGQ>(A, d, c_lds, f0_lds, f1_lds, a0_lds, a1_lds);
    } else {
        const int32_t xcd = blockIdx.x & 7;
        for (;;) {
            int32_t i = 0;
            if (threadIdx.x == 0) i = atomicAdd(&A.claim[xcd], 1);
            i = __shfl(i, 0);
            if (i >= A.docs_per_xcd) break;
            const int32_t d = xcd * A.docs_per_xcd + i;
            if (d >= A.D) break;
            sample_doc_assoc<KPL, SP, WIDE, BIGQ>(A, d, c_lds, f0_lds, f1_lds, a0_lds, a1_lds);
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

template <int KPL, int SP>
hipError_t launch_assoc_kpl(const AssocArgs &A, hipStream_t st)
{
    const unsigned grid = (unsigned)(8 * A.docs_per_xcd);
    // the persistent launch: at most one workgroup per wavefront slot
    const unsigned pgrid = grid < 4096u ? grid : 4096u;
    if (A.nQ > kSmallQ) {
        hipLaunchKernelGGL((k_sample_assoc<KPL, SP, false, true>), dim3(grid), dim3(64), 0, st, A);
        hipLaunchKernelGGL((k_sample_assoc<KPL, SP, true, true>), dim3(pgrid), dim3(64), 0, st, A);
    } else {
        hipLaunchKernelGGL((k_sample_assoc<KPL, SP, false, false>), dim3(grid), dim3(64), 0, st, A);
        hipLaunchKernelGGL((k_sample_assoc<KPL, SP, true, false>), dim3(pgrid), dim3(64), 0, st, A);
    }
    return hipGetLastError();
}

template <int SP>
hipError_t launch_assoc_sp(const AssocArgs &A, int kpl, hipStream_t st)
{
    switch (kpl) {
    case 1: return launch_assoc_kpl<1, SP>(A, st);
    case 2: return launch_assoc_kpl<2, SP>(A, st);
    case 4: return launch_assoc_kpl<4, SP>(A, st);
    case 8: return launch_assoc_kpl<8, SP>(A, st);
    case 12: return launch_assoc_kpl<12, SP>(A, st);
    default: return launch_assoc_kpl<16, SP>(A, st);
    }
}

}  // namespace

hipError_t launch_sample_assoc(const Model &m, const DeviceBuffers &b, const int32_t *zr_old,
                               int32_t *zr_new, uint32_t sweep, uint64_t seed, float *tr_w,
                               float *tr_u, int64_t tr_begin, int64_t tr_end, hipStream_t st)
{
    if (m.D <= 0 || m.N <= 0) return hipSuccess;
    AssocArgs A;
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
    A.srcrec = b.srcrec;
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
    A.S = m.S;
    A.nQ = tri_index(m.ncap, 0);
    A.GK = (int64_t)m.G * m.Kp;
    A.docs_per_xcd = (m.D + 7) / 8;
    A.sweep = sweep;
    A.alpha = (float)m.alpha;
    A.gamma = (float)m.gamma;
    const int kpl = sampler_kpl(m.K);
    switch (m.Sp) {
    case 1: return launch_assoc_sp<1>(A, kpl, st);
    case 2: return launch_assoc_sp<2>(A, kpl, st);
    case 4: return launch_assoc_sp<4>(A, kpl, st);
    case 8: return launch_assoc_sp<8>(A, kpl, st);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace spdp
