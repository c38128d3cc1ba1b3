// spdp_internal.hpp -- device-side data layout, helpers and kernel launchers
// shared by the translation units of the gfx950 SPDP library.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/spdp.h"

namespace spdp {

// ---------------------------------------------------------------------------
// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11).  Counter (token lo, token
// hi, sweep, purpose), key = seed.  Only word 0 of each block is used.
// ---------------------------------------------------------------------------
enum : uint32_t { kPurposeSample = 0u, kPurposeInit = 1u };

__host__ __device__ __forceinline__ uint32_t philox_x0(uint64_t seed, uint64_t ctr_lo64,
                                                       uint32_t c2, uint32_t c3)
{
    uint32_t x0 = (uint32_t)ctr_lo64, x1 = (uint32_t)(ctr_lo64 >> 32), x2 = c2, x3 = c3;
    uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        const uint64_t p0 = (uint64_t)0xD2511F53u * x0;
        const uint64_t p1 = (uint64_t)0xCD9E8D57u * x2;
        const uint32_t y0 = (uint32_t)(p1 >> 32) ^ x1 ^ k0;
        const uint32_t y1 = (uint32_t)p1;
        const uint32_t y2 = (uint32_t)(p0 >> 32) ^ x3 ^ k1;
        const uint32_t y3 = (uint32_t)p0;
        x0 = y0; x1 = y1; x2 = y2; x3 = y3;
        k0 += 0x9E3779B9u;
        k1 += 0xBB67AE85u;
    }
    return x0;
}

// ---------------------------------------------------------------------------
// Division of a non-negative int32 by a runtime constant d (1 <= d < 2^31) by
// multiply-shift: q = (n * m) >> s with m = ceil(2^s / d), s = 31 + ceil(log2 d).
// Exact for 0 <= n < 2^31 because n * (m d - 2^s) < 2^31 * d <= 2^s; m <= 2^32 + 1
// so the 64-bit product n * m cannot overflow.
// ---------------------------------------------------------------------------
struct FastDiv {
    uint64_t m;
    uint32_t s;
};

inline FastDiv make_fastdiv(uint32_t d)
{
    uint32_t l = 0;
    while ((1ull << l) < d) ++l;
    FastDiv f;
    f.s = 31 + l;
    f.m = (uint64_t)((((unsigned __int128)1 << f.s) + d - 1) / d);
    return f;
}

__host__ __device__ __forceinline__ uint32_t fastdiv(uint32_t n, FastDiv f)
{
    return (uint32_t)(((uint64_t)n * f.m) >> f.s);
}

// Packed per-token state: zr = 2 z + r, plus (model with word associations)
// the slot s of a head's source word in bits 16..18: zr = s << 16 | 2 z + r.
// A token with r = 0 has s = 0, and the plain model has s = 0 throughout.
constexpr int32_t kSlotShift = 16;
__host__ __device__ __forceinline__ int32_t zr_pack(int32_t z, int32_t r) { return 2 * z + r; }
__host__ __device__ __forceinline__ int32_t zr_pack(int32_t z, int32_t r, int32_t s)
{
    return (s << kSlotShift) | (2 * z + r);
}
__host__ __device__ __forceinline__ int32_t zr_topic(int32_t v) { return (v & 0xFFFF) >> 1; }
__host__ __device__ __forceinline__ int32_t zr_slot(int32_t v) { return v >> kSlotShift; }

// Index of (n, t) in a lower-triangular table with row n at n (n + 1) / 2.
__host__ __device__ __forceinline__ int64_t tri_index(int64_t n, int64_t t)
{
    return n * (n + 1) / 2 + t;
}

// ---------------------------------------------------------------------------
// Device state.  Count rows: row index q = g V + w; row q of nt holds the Kp
// topic cells of (g, w) (Kp = K rounded up to the sampler's vector width,
// padding cells stay zero), each cell packing the customer count n in bits
// 0..15 and the table count t in bits 16..31.  B rows are indexed by w.
// ---------------------------------------------------------------------------
constexpr int32_t kCountBits = 16;
constexpr int32_t kCountMax = (1 << kCountBits) - 1;  // largest n a packed cell holds

// Narrow rows.  A (group, word) pair with at most kNarrowMax tokens in the
// corpus can never have a count above kNarrowMax in any state (n[g][k][w] <=
// c[g][w]), so its row also exists as 16-bit cells n | t << 8, half the
// bytes, which the samplers read instead.  Which rows are narrow is fixed at
// creation; the rebuild writes only the 16-bit copy of a narrow row, and its
// 32-bit row is rewritten from that copy when an entry point reads it.
constexpr int32_t kNarrowMax = 255;
__host__ __device__ __forceinline__ uint16_t narrow_of(int32_t packed)
{
    return (uint16_t)((packed & 0xFF) | ((packed >> kCountBits) << 8));
}
__host__ __device__ __forceinline__ int32_t wide_of(uint32_t cell16)
{
    return (int32_t)((cell16 & 0xFFu) | ((cell16 & 0xFF00u) << 8));
}

struct Model {
    int64_t N;
    int32_t D, V, G, K, Kp;
    float alpha_f, a_f, b_f, gamma_f, Vgamma_f;
    double alpha, a, b, gamma;
    int32_t ncap;  // largest per-(g, w) token count: every n' < ncap in a sweep
    FastDiv divV;  // q -> g
    // word associations (0 for the plain model, P = I): S = longest source
    // list, Sp = S rounded up to 1, 2, 4 or 8 (the slot count of the records)
    int32_t S = 0, Sp = 0;
};

// Inputs of the sampler's rare fp64 re-decision path, kept in device memory
// so that they occupy no scalar registers on the common path.
struct ExactCtx {
    const int32_t *Ngk, *Tgk, *Bk, *B;
    const double *logS;
    const double2 *Q64;  // [tri(ncap)] fp64 (Q0, Q1) ratio pairs
    double a, b, Vgamma, alpha, gamma;
    int32_t K, ncap;
    // word associations: source records and fp64 p of each row (Sp slots)
    const int32_t *srcrec;
    const double *p64;
    int32_t Sp;
};

struct DeviceBuffers {
    int32_t *gw = nullptr;        // [N]  row index g V + w of each token
    int64_t *doc_off = nullptr;   // [D+1]
    int32_t *doc_group = nullptr; // [D]
    int32_t *zr[2] = {nullptr, nullptr}; // [N] current / next packed state
    int32_t *nt = nullptr;        // [G V][Kp] packed n | t << 16
    uint16_t *nt16 = nullptr;     // [G V][Kp] narrow rows as n | t << 8 (other rows unused);
                                  // the rebuild writes a narrow row only here
    uint8_t *row_narrow = nullptr; // [G V] 1 if row q is narrow (c[g][w] <= kNarrowMax)
    uint8_t *tok_narrow = nullptr; // [N] row_narrow of each token's row (the sampler's stream)
    int32_t *B = nullptr;         // [V][Kp]   shadow-base table counts
    uint16_t *B16 = nullptr;      // [V][Kp]   min(B, 65535): the sampler's copy
    int32_t *wide = nullptr;      // [1] 1 if some B exceeds 65535 (the sampler then reads B)
    int32_t *claim = nullptr;     // [9] documents claimed per XCD by the samplers' persistent
                                  // launch (32-bit shadow-base rows) and its finished
                                  // workgroups; zero between launches (its last workgroup
                                  // clears them)
    int32_t *perm = nullptr;      // [N] tokens grouped by row (any order inside a row)
    int32_t *row_off = nullptr;   // [G V + 1] offsets of each row's tokens in perm
    int32_t *tok_slot = nullptr;  // [N] each token's slot in the routed state copy zr_b
    int32_t *row_slot = nullptr;  // [N] the slot of row list entry j: tok_slot[perm[j]]
    uint16_t *zr_b = nullptr;     // [N] the states routed by row bucket, as 16 bits (a state
                                  // without a source slot is z << 1 | r < 2^11), rewritten
                                  // by every rebuild before it gathers from them (plain
                                  // model only: null with word associations)
    int32_t *Ngk = nullptr;       // [G][Kp]
    int32_t *Tgk = nullptr;       // [G][Kp]
    int32_t *Bk = nullptr;        // [Kp]
    float *f0 = nullptr;          // [G][Kp] 1 / (b + N_gk)
    float *f1 = nullptr;          // [G][Kp] (b + a T_gk) / (b + N_gk) / (V gamma + B_k)
    float *fk = nullptr;          // [3][G][Kp] the same with one customer removed:
                                  //   1/(b + N - 1), and f1 for a removed non-head / head
    float2 *Q = nullptr;          // [tri(ncap)] (Q0, Q1) folded Stirling ratios
    double *logS = nullptr;       // [tri(ncap + 1)] log S^n_{t,a}
    double2 *Q64 = nullptr;       // [tri(ncap)] the ratio pairs in fp64
    double *lfact = nullptr;      // [ncap + 1] log n!
    uint32_t *rep_part = nullptr; // [G V] heads promoted per row in the last rebuild
    unsigned long long *part = nullptr; // reduction partials
    unsigned long long *ctr = nullptr;  // [4] changed, repaired (filled on demand)
    double *partial = nullptr;    // loglik block partials
    int64_t partial_len = 0;
    int32_t *err = nullptr;       // [2] device error flags
    double *scalar = nullptr;     // [1] reduction result
    ExactCtx *exact = nullptr;    // [1] the sampler's fp64 re-decision inputs
    // debug-conditional buffers (allocated on demand)
    int32_t *zr_dbg = nullptr;
    float *tr_w = nullptr;
    float *tr_u = nullptr;
    int64_t tr_cap = 0;
    // word associations (allocated only for that model): per row q = g V + w,
    // the Sp source words followed by their p in fp32 (a padding slot repeats
    // the first source with p = 0), the same p in fp64, and the slot a head
    // promoted by the repair takes (the most probable source, first on ties)
    int32_t *srcrec = nullptr;    // [G V][2 Sp]
    double *p64 = nullptr;        // [G V][Sp]
    uint8_t *head_slot = nullptr; // [G V]
    // asynchronous sweep (allocated on its first use): visiting order of the
    // word order rearrangement, document of each token, live document counts
    int32_t *order = nullptr;     // [N]
    int32_t *tok_doc = nullptr;   // [N]
    int32_t *cdk = nullptr;       // [D][Kp]
};

// ---------------------------------------------------------------------------
// Kernel launchers (each returns hipSuccess or the launch error).
// ---------------------------------------------------------------------------
hipError_t launch_fill_i32(int32_t *p, int64_t n, int32_t v, hipStream_t st);
hipError_t launch_fill_u32(uint32_t *p, int64_t n, uint32_t v, hipStream_t st);
hipError_t launch_fill_u64(unsigned long long *p, int64_t n, unsigned long long v, hipStream_t st);
hipError_t launch_make_gw(const Model &m, const int32_t *words, const int64_t *doc_off,
                          const int32_t *doc_group, int32_t *gw, int32_t *gw_count,
                          int32_t *bad, hipStream_t st);
hipError_t launch_max_i32(const int32_t *x, int64_t n, int32_t *out, hipStream_t st);
// narrow-row flags from the per-row token counts: per row and per token; the
// number of narrow rows is added to *n_narrow
hipError_t launch_narrow_flags(const Model &m, const int32_t *gw, const int32_t *gw_count,
                               uint8_t *row_narrow, uint8_t *tok_narrow,
                               unsigned long long *n_narrow, hipStream_t st);
hipError_t launch_stirling(const Model &m, double *logS, float2 *Q, double2 *Q64, double *lfact,
                           hipStream_t st);
hipError_t launch_init_z(const Model &m, uint64_t seed, int32_t *zr, hipStream_t st);
hipError_t launch_pack_zr(const Model &m, const int32_t *z, const uint8_t *r, int32_t *zr,
                          int32_t *bad, hipStream_t st);
hipError_t launch_unpack_zr(const Model &m, const int32_t *zr, int32_t *z, uint8_t *r,
                            hipStream_t st);
hipError_t build_row_index(const Model &m, DeviceBuffers &b, const int32_t *gw_count,
                           hipStream_t st);
// count rows with the repair, and the shadow-base counts B (zeroed, then each
// row's table counts added) of the plain model, from the state zr
hipError_t launch_rows(const Model &m, const DeviceBuffers &b, int32_t *zr, hipStream_t st);
// the 32-bit rows of the narrow rows from their 16-bit copies (the rebuild
// writes a narrow row only as its copy; entry points that read 32-bit rows
// call this first)
hipError_t launch_widen(const Model &m, const DeviceBuffers &b, hipStream_t st);
// word associations: count rows with the repair, and the shadow-base counts
// keyed by source (B zeroed, then one increment per head)
hipError_t launch_rows_assoc(const Model &m, const DeviceBuffers &b, int32_t *zr, hipStream_t st);
// B16 and the width flag from B (after either rebuild)
hipError_t launch_base16(const Model &m, const DeviceBuffers &b, hipStream_t st);
hipError_t launch_pack_zrs(const Model &m, const DeviceBuffers &b, const int32_t *z,
                           const uint8_t *r, const uint8_t *s, int32_t *zr, int32_t *bad,
                           hipStream_t st);
hipError_t launch_unpack_slot(const Model &m, const int32_t *zr, uint8_t *s, hipStream_t st);
hipError_t launch_unpack_counts(const Model &m, const DeviceBuffers &b, int32_t g,
                                int32_t *n_out, int32_t *t_out, hipStream_t st);
// invariant check of the count state (count rows, in the copy the rebuild
// writes, against a recount of the tokens' states; the shadow base; the
// totals): the number of failing cells or totals is added to *bad
hipError_t launch_check(const Model &m, const DeviceBuffers &b, const int32_t *zr,
                        int32_t *scratch_totals, unsigned long long *bad, hipStream_t st);
hipError_t launch_stat_sums(const Model &m, const DeviceBuffers &b, const int32_t *zr_now,
                            const int32_t *zr_before, hipStream_t st);
int64_t stat_partials_needed();
hipError_t launch_totals(const Model &m, const DeviceBuffers &b, const int32_t *zr,
                         hipStream_t st);
// the same into other arrays (N, T: [G][Kp], Bk: [Kp])
hipError_t launch_totals_into(const Model &m, const DeviceBuffers &b, const int32_t *zr,
                              int32_t *Ngk, int32_t *Tgk, int32_t *Bk, hipStream_t st);
hipError_t launch_factors(const Model &m, const DeviceBuffers &b, hipStream_t st);
hipError_t launch_sample(const Model &m, const DeviceBuffers &b, const int32_t *zr_old,
                         int32_t *zr_new, uint32_t sweep, uint64_t seed, float *tr_w,
                         float *tr_u, int64_t tr_begin, int64_t tr_end, hipStream_t st);
hipError_t launch_sample_assoc(const Model &m, const DeviceBuffers &b, const int32_t *zr_old,
                               int32_t *zr_new, uint32_t sweep, uint64_t seed, float *tr_w,
                               float *tr_u, int64_t tr_begin, int64_t tr_end, hipStream_t st);
hipError_t launch_loglik(const Model &m, const DeviceBuffers &b, const int32_t *zr,
                         hipStream_t st);
// asynchronous sweep: token -> document and position, the visiting order
// (stable sort of tokens by position inside the document), document counts,
// the sampling pass with live atomics (waves wavefronts)
hipError_t launch_tok_doc(const Model &m, const int64_t *doc_off, int32_t *tok_doc, int32_t *pos,
                          hipStream_t st);
hipError_t build_visit_order(const Model &m, DeviceBuffers &b, hipStream_t st);
hipError_t launch_doc_counts(const Model &m, const DeviceBuffers &b, const int32_t *zr,
                             int32_t *cdk, hipStream_t st);
hipError_t launch_sample_async(const Model &m, const DeviceBuffers &b, const int32_t *order,
                               const int32_t *tok_doc, int32_t *cdk, int32_t *zr, uint32_t sweep,
                               uint64_t seed, int32_t waves, bool live_totals, hipStream_t st);
int64_t loglik_partials_needed();

hipError_t launch_theta(const Model &m, const DeviceBuffers &b, const int32_t *zr, double *theta,
                        hipStream_t st);
hipError_t launch_phi0(const Model &m, const DeviceBuffers &b, double *phi0, hipStream_t st);
hipError_t launch_phig(const Model &m, const DeviceBuffers &b, int32_t g, double *phi,
                       hipStream_t st);
hipError_t launch_foldin(const Model &m, const DeviceBuffers &b, int32_t D_test,
                         const int32_t *gw, const int64_t *doc_off, const int32_t *doc_group,
                         int32_t n_sweeps, uint64_t seed, int32_t *z, double *ll_doc,
                         hipStream_t st);

// Hellinger distances between the topics of two models (P [V][kp], Q [V][kq],
// topics contiguous): the launch shape and the partial-sum buffer it needs
// (slices * kp * kq doubles).
struct HellingerPlan {
    int64_t slice = 0;   // outcomes per slice (a multiple of the LDS stage)
    int32_t slices = 1;  // outcome slices (grid y)
    int32_t tiles_j = 1; // 64-wide tiles along kq
    int64_t tiles = 1;   // output tiles (grid x)
};
HellingerPlan hellinger_plan(int32_t kp, int32_t kq, int64_t V);
// the same with at most max_part partial sums (slices * kp * kq <= max_part
// whenever kp * kq <= max_part)
HellingerPlan hellinger_plan(int32_t kp, int32_t kq, int64_t V, int64_t max_part);
// The allocation-free variant's partial-sum buffer: a file-scope device array
// of kHellingerScratch doubles (8 MiB) per GPU; hellinger_scratch() returns
// its device address on `device`, looked up once per device (a hipError_t).
constexpr int64_t kHellingerScratch = 1 << 20;
constexpr int kMaxDevices = 64;
int hellinger_scratch(int device, double **out);
hipError_t launch_hellinger(const HellingerPlan &p, const double *P, int32_t kp, const double *Q,
                            int32_t kq, int64_t V, double *part, double *h, hipStream_t st);
// least-total-cost matching of the rows of c [kp][kq] (kp <= kq, finite):
// match[i] = column of row i; returns the total cost (host code)
double align_topics_host(const double *c, int32_t kp, int32_t kq, int32_t *match);

// The sampler's per-lane topic count for K topics (4 at most per dwordx4).
hipError_t launch_read_probe(const void *buf, int64_t bytes, int32_t row_bytes, int64_t rows,
                             int32_t waves, hipStream_t st);
int sampler_kpl(int32_t K);
int32_t padded_K(int32_t K);

}  // namespace spdp
