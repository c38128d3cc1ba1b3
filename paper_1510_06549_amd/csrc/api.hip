// api.hip -- the extern "C" boundary (declared in include/spdp.h): argument
// validation, device memory, error mapping and the order of kernel launches.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "spdp_internal.hpp"

using namespace spdp;

namespace {

thread_local std::string g_last_error;

int fail(int code, const char *fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return code;
}

#define HIP_TRY(expr)                                                                      \
    do {                                                                                   \
        hipError_t e_ = (expr);                                                            \
        if (e_ != hipSuccess)                                                              \
            return fail(SPDP_E_HIP, "%s failed: %s", #expr, hipGetErrorString(e_));        \
    } while (0)

constexpr int64_t kStirlingBudget = 72ll << 30;  // bytes for log S + fp32 and fp64 ratio pairs
// The cache covers every n the packed counts can hold (68.7 GB of tables at
// ncap = 65535); past 2^29 fp32 ratio pairs (ncap > 32767) the samplers
// address them with 64-bit instead of 32-bit offsets.
constexpr int32_t kMaxNcap = kCountMax;

struct EventPair {
    hipEvent_t a, b;
};

}  // namespace

struct spdp_state {
    Model m{};
    DeviceBuffers b{};
    hipStream_t st = nullptr;
    int device = 0;
    int cur = 0;
    int64_t bytes = 0;
    int64_t n_narrow_rows = 0;
    // true while the 32-bit rows of the narrow rows equal their 16-bit copies
    // (the rebuild writes a narrow row only as its copy)
    mutable bool rows32 = false;
    bool timing = false;
    std::vector<EventPair> events[SPDP_NKERNELS];
    std::vector<void *> allocs;
};

namespace {

template <typename T>
int dev_alloc(spdp_state *s, T **p, int64_t count, const char *what)
{
    *p = nullptr;
    if (count <= 0) count = 1;
    const size_t bytes = (size_t)count * sizeof(T);
    void *q = nullptr;
    hipError_t e = hipMalloc(&q, bytes);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        return fail(SPDP_E_NOMEM, "hipMalloc of %zu bytes for %s failed: %s", bytes, what,
                    hipGetErrorString(e));
    }
    s->allocs.push_back(q);
    s->bytes += (int64_t)bytes;
    *p = static_cast<T *>(q);
    return SPDP_OK;
}

void free_state(spdp_state *s)
{
    if (!s) return;
    (void)hipSetDevice(s->device);
    if (s->st) (void)hipStreamSynchronize(s->st);
    else (void)hipDeviceSynchronize();
    for (void *p : s->allocs) (void)hipFree(p);
    if (s->b.zr_dbg) (void)hipFree(s->b.zr_dbg);
    if (s->b.tr_w) (void)hipFree(s->b.tr_w);
    if (s->b.tr_u) (void)hipFree(s->b.tr_u);
    for (auto &v : s->events)
        for (auto &ev : v) {
            (void)hipEventDestroy(ev.a);
            (void)hipEventDestroy(ev.b);
        }
    delete s;
}

int sync(const spdp_state *s)
{
    HIP_TRY(hipStreamSynchronize(s->st));
    return SPDP_OK;
}

// Run `launch` with optional event timing of kernel class `cls`.
template <typename F>
int timed(spdp_state *s, int cls, F launch)
{
    EventPair ev{};
    if (s->timing) {
        HIP_TRY(hipEventCreate(&ev.a));
        HIP_TRY(hipEventCreate(&ev.b));
        HIP_TRY(hipEventRecord(ev.a, s->st));
    }
    HIP_TRY(launch());
    if (s->timing) {
        HIP_TRY(hipEventRecord(ev.b, s->st));
        s->events[cls].push_back(ev);
    }
    return SPDP_OK;
}

// Counts (with the repair of every cell left without a table), shadow base
// and totals for the packed state in zr[cur]; the other state buffer gets a
// copy so that the statistics of a fresh state read zero.
int rebuild_state(spdp_state *s)
{
    const Model &m = s->m;
    DeviceBuffers &b = s->b;
    int32_t *zr = b.zr[s->cur];
    if (m.Sp > 0) HIP_TRY(launch_rows_assoc(m, b, zr, s->st));
    else HIP_TRY(launch_rows(m, b, zr, s->st));
    HIP_TRY(launch_base16(m, b, s->st));
    s->rows32 = false;
    HIP_TRY(launch_totals(m, b, zr, s->st));
    if (m.N > 0)
        HIP_TRY(hipMemcpyAsync(b.zr[1 - s->cur], zr, (size_t)m.N * sizeof(int32_t),
                               hipMemcpyDeviceToDevice, s->st));
    return SPDP_OK;
}

// The 32-bit rows of the narrow rows, rewritten from their 16-bit copies once
// after each rebuild, for the entry points that read 32-bit rows (export,
// estimates, likelihood, fold-in, the asynchronous sweep).
hipError_t widen_rows(const spdp_state *s)
{
    if (s->rows32) return hipSuccess;
    hipError_t e = launch_widen(s->m, s->b, s->st);
    if (e == hipSuccess) s->rows32 = true;
    return e;
}

int check_device_flags(spdp_state *s, int32_t *host_err)
{
    HIP_TRY(hipMemcpyAsync(host_err, s->b.err, 2 * sizeof(int32_t), hipMemcpyDeviceToHost, s->st));
    return sync(s);
}

// Word associations: validate the source lists of the G V rows and build the
// padded device records (Sp slots per row; a padding slot repeats the row's
// first source with p = 0), the fp64 p and the repair's head slot per row.
int check_assoc(const spdp_assoc *A, int32_t G, int32_t V)
{
    if (A->max_sources < 1 || A->max_sources > SPDP_MAX_SOURCES)
        return fail(SPDP_E_ARG, "max_sources must be in [1, %d]", SPDP_MAX_SOURCES);
    if (!A->row_off || !A->src || !A->p) return fail(SPDP_E_ARG, "null association array");
    const int64_t rows = (int64_t)G * V;
    if (A->row_off[0] != 0) return fail(SPDP_E_ARG, "association row_off must start at 0");
    int32_t longest = 0;
    for (int64_t q = 0; q < rows; ++q) {
        const int64_t b0 = A->row_off[q], b1 = A->row_off[q + 1];
        if (b1 <= b0) return fail(SPDP_E_ARG, "association row %lld has no source", (long long)q);
        if (b1 - b0 > A->max_sources)
            return fail(SPDP_E_ARG, "association row %lld lists more than max_sources sources",
                        (long long)q);
        longest = std::max<int32_t>(longest, (int32_t)(b1 - b0));
        for (int64_t e = b0; e < b1; ++e) {
            if (A->src[e] < 0 || A->src[e] >= V)
                return fail(SPDP_E_ARG, "association source out of [0, vocab) in row %lld",
                            (long long)q);
            if (!(A->p[e] > 0.0) || !std::isfinite(A->p[e]))
                return fail(SPDP_E_ARG, "association p must be finite and > 0 (row %lld)",
                            (long long)q);
            for (int64_t f = b0; f < e; ++f)
                if (A->src[f] == A->src[e])
                    return fail(SPDP_E_ARG, "association row %lld repeats source %d",
                                (long long)q, A->src[e]);
        }
    }
    if (longest != A->max_sources)
        return fail(SPDP_E_ARG, "max_sources (%d) is not the longest row (%d)", A->max_sources,
                    longest);
    return SPDP_OK;
}

int upload_assoc(spdp_state *s, const spdp_assoc *A)
{
    Model &m = s->m;
    DeviceBuffers &B = s->b;
    m.S = A->max_sources;
    m.Sp = m.S <= 1 ? 1 : (m.S <= 2 ? 2 : (m.S <= 4 ? 4 : 8));
    const int64_t rows = (int64_t)m.G * m.V;
    std::vector<int32_t> rec((size_t)(rows * 2 * m.Sp));
    std::vector<double> p64((size_t)(rows * m.Sp), 0.0);
    std::vector<uint8_t> hs((size_t)rows);
    for (int64_t q = 0; q < rows; ++q) {
        const int64_t b0 = A->row_off[q], n = A->row_off[q + 1] - b0;
        int32_t *r = rec.data() + q * 2 * m.Sp;
        int32_t best = 0;
        for (int32_t sl = 0; sl < m.Sp; ++sl) {
            const bool real = sl < n;
            const float pf = real ? (float)A->p[b0 + sl] : 0.0f;
            r[sl] = A->src[b0 + (real ? sl : 0)];
            std::memcpy(&r[m.Sp + sl], &pf, sizeof pf);
            p64[(size_t)(q * m.Sp + sl)] = real ? A->p[b0 + sl] : 0.0;
            if (real && A->p[b0 + sl] > A->p[b0 + best]) best = sl;
        }
        hs[(size_t)q] = (uint8_t)best;
    }
    int rc;
    if ((rc = dev_alloc(s, &B.srcrec, rows * 2 * m.Sp, "association records")) != SPDP_OK) return rc;
    if ((rc = dev_alloc(s, &B.p64, rows * m.Sp, "association p")) != SPDP_OK) return rc;
    if ((rc = dev_alloc(s, &B.head_slot, rows, "head slots")) != SPDP_OK) return rc;
    HIP_TRY(hipMemcpyAsync(B.srcrec, rec.data(), rec.size() * sizeof(int32_t),
                           hipMemcpyHostToDevice, s->st));
    HIP_TRY(hipMemcpyAsync(B.p64, p64.data(), p64.size() * sizeof(double), hipMemcpyHostToDevice,
                           s->st));
    HIP_TRY(hipMemcpyAsync(B.head_slot, hs.data(), hs.size(), hipMemcpyHostToDevice, s->st));
    return sync(s);  // the host vectors go out of scope
}

int create_state(const spdp_corpus *corpus, const spdp_groups *groups, const spdp_assoc *assoc,
                 int32_t K, double alpha, double a, double b, double gamma, spdp_state **out);

}  // namespace

extern "C" {

const char *spdp_last_error(void) { return g_last_error.c_str(); }

int spdp_create(const spdp_corpus *corpus, const spdp_groups *groups, int32_t K, double alpha,
                double a, double b, double gamma, spdp_state **out)
{
    g_last_error.clear();
    return create_state(corpus, groups, nullptr, K, alpha, a, b, gamma, out);
}

int spdp_create_assoc(const spdp_corpus *corpus, const spdp_groups *groups,
                      const spdp_assoc *assoc, int32_t K, double alpha, double a, double b,
                      double gamma, spdp_state **out)
{
    g_last_error.clear();
    if (!assoc) return fail(SPDP_E_ARG, "assoc is NULL");
    return create_state(corpus, groups, assoc, K, alpha, a, b, gamma, out);
}

}  // extern "C"

namespace {

int create_state(const spdp_corpus *corpus, const spdp_groups *groups, const spdp_assoc *assoc,
                 int32_t K, double alpha, double a, double b, double gamma, spdp_state **out)
{
    if (!out) return fail(SPDP_E_ARG, "out is NULL");
    *out = nullptr;
    if (!corpus || !groups) return fail(SPDP_E_ARG, "corpus or groups is NULL");
    const int64_t N = corpus->n_tokens;
    const int32_t D = corpus->n_docs, V = corpus->vocab, G = groups->n_groups;
    if (N < 0 || N >= (1ll << 31)) return fail(SPDP_E_ARG, "n_tokens %lld out of [0, 2^31)", (long long)N);
    if (D < 1) return fail(SPDP_E_ARG, "n_docs must be >= 1");
    if (V < 1) return fail(SPDP_E_ARG, "vocab must be >= 1");
    if (G < 1) return fail(SPDP_E_ARG, "n_groups must be >= 1");
    if ((int64_t)G * V >= (1ll << 31)) return fail(SPDP_E_ARG, "n_groups * vocab must be < 2^31");
    if (K < 1 || K > SPDP_MAX_K) return fail(SPDP_E_ARG, "K must be in [1, %d]", SPDP_MAX_K);
    if (!(alpha > 0.0) || !std::isfinite(alpha)) return fail(SPDP_E_ARG, "alpha must be > 0");
    if (!(gamma > 0.0) || !std::isfinite(gamma)) return fail(SPDP_E_ARG, "gamma must be > 0");
    if (!(a >= 0.0 && a < 1.0)) return fail(SPDP_E_ARG, "discount a must be in [0, 1)");
    if (!(b > 0.0) || !std::isfinite(b)) return fail(SPDP_E_ARG, "concentration b must be > 0");
    if (!corpus->doc_offsets || !groups->doc_group || (N > 0 && !corpus->words))
        return fail(SPDP_E_ARG, "null corpus array");
    const int64_t *off = corpus->doc_offsets;
    if (off[0] != 0 || off[D] != N) return fail(SPDP_E_ARG, "doc_offsets must start at 0 and end at N");
    for (int32_t d = 0; d < D; ++d)
        if (off[d + 1] < off[d]) return fail(SPDP_E_ARG, "doc_offsets not nondecreasing at %d", d);
    if (assoc) {
        const int rca = check_assoc(assoc, G, V);
        if (rca != SPDP_OK) return rca;
    }

    spdp_state *s = new (std::nothrow) spdp_state();
    if (!s) return fail(SPDP_E_NOMEM, "host allocation failed");
    int rc = SPDP_OK;
#define TRY(x)                          \
    do {                                \
        if ((rc = (x)) != SPDP_OK) {    \
            std::string msg_ = g_last_error; \
            free_state(s);              \
            g_last_error = msg_;        \
            return rc;                  \
        }                               \
    } while (0)
#define TRY_HIP(x)                                                                         \
    do {                                                                                   \
        hipError_t e_ = (x);                                                               \
        if (e_ != hipSuccess) {                                                            \
            fail(SPDP_E_HIP, "%s failed: %s", #x, hipGetErrorString(e_));                  \
            std::string msg_ = g_last_error;                                               \
            free_state(s);                                                                 \
            g_last_error = msg_;                                                           \
            return SPDP_E_HIP;                                                             \
        }                                                                                  \
    } while (0)

    TRY_HIP(hipGetDevice(&s->device));
    s->st = (hipStream_t)corpus->hip_stream;
    {
        // the allocation-free Hellinger's scratch address on this device
        double *scratch_addr = nullptr;
        TRY_HIP((hipError_t)hellinger_scratch(s->device, &scratch_addr));
    }
    Model &m = s->m;
    m.N = N;
    m.D = D;
    m.V = V;
    m.G = G;
    m.K = K;
    m.Kp = padded_K(K);
    m.alpha = alpha;
    m.a = a;
    m.b = b;
    m.gamma = gamma;
    m.alpha_f = (float)alpha;
    m.a_f = (float)a;
    m.b_f = (float)b;
    m.gamma_f = (float)gamma;
    m.Vgamma_f = (float)((double)V * gamma);
    m.divV = make_fastdiv((uint32_t)V);
    DeviceBuffers &B = s->b;
    const int64_t rows = (int64_t)G * V;

    // corpus
    int32_t *words_d = nullptr, *gw_count = nullptr;
    TRY(dev_alloc(s, &B.gw, N, "token rows"));
    TRY(dev_alloc(s, &B.doc_off, (int64_t)D + 1, "doc offsets"));
    TRY(dev_alloc(s, &B.doc_group, D, "doc groups"));
    TRY(dev_alloc(s, &B.err, 2, "error flags"));
    TRY(dev_alloc(s, &B.ctr, 4, "counters"));
    TRY(dev_alloc(s, &B.claim, 9, "document claims"));
    TRY_HIP(launch_fill_i32(B.claim, 9, 0, s->st));
    TRY(dev_alloc(s, &B.scalar, 1, "scalar"));
    TRY_HIP(launch_fill_i32(B.err, 2, 0, s->st));
    {
        void *tmp = nullptr;
        if (hipMalloc(&tmp, (size_t)(N > 0 ? N : 1) * sizeof(int32_t)) != hipSuccess) {
            (void)hipGetLastError();
            TRY(fail(SPDP_E_NOMEM, "staging buffer for words"));
        }
        words_d = (int32_t *)tmp;
        if (hipMalloc(&tmp, (size_t)(rows + 1) * sizeof(int32_t)) != hipSuccess) {
            (void)hipGetLastError();
            (void)hipFree(words_d);
            TRY(fail(SPDP_E_NOMEM, "staging buffer for word counts"));
        }
        gw_count = (int32_t *)tmp;
    }
    auto cleanup_staging = [&]() {
        (void)hipFree(words_d);
        (void)hipFree(gw_count);
    };
    hipError_t e = hipSuccess;
    if (N > 0)
        e = hipMemcpyAsync(words_d, corpus->words, (size_t)N * sizeof(int32_t),
                           hipMemcpyHostToDevice, s->st);
    if (e == hipSuccess)
        e = hipMemcpyAsync(B.doc_off, off, (size_t)(D + 1) * sizeof(int64_t), hipMemcpyHostToDevice,
                           s->st);
    if (e == hipSuccess)
        e = hipMemcpyAsync(B.doc_group, groups->doc_group, (size_t)D * sizeof(int32_t),
                           hipMemcpyHostToDevice, s->st);
    if (e == hipSuccess) e = launch_fill_i32(gw_count, rows + 1, 0, s->st);
    if (e == hipSuccess) e = launch_make_gw(m, words_d, B.doc_off, B.doc_group, B.gw, gw_count, B.err, s->st);
    if (e == hipSuccess) e = launch_max_i32(gw_count, rows, B.err + 1, s->st);
    int32_t herr[2] = {0, 0};
    if (e == hipSuccess) e = hipMemcpyAsync(herr, B.err, sizeof herr, hipMemcpyDeviceToHost, s->st);
    if (e == hipSuccess) e = hipStreamSynchronize(s->st);
    if (e != hipSuccess) cleanup_staging();
    TRY_HIP(e);
    if ((herr[0] & 3) || herr[1] > kCountMax) cleanup_staging();
    if (herr[0] & 1) TRY(fail(SPDP_E_ARG, "doc_group out of [0, n_groups)"));
    if (herr[0] & 2) TRY(fail(SPDP_E_ARG, "word id out of [0, vocab)"));
    if (herr[1] > kCountMax)
        TRY(fail(SPDP_E_RANGE, "a (group, word) pair occurs %d times; packed counts hold %d",
                 herr[1], kCountMax));
    m.ncap = herr[1] < 1 ? 1 : herr[1];
    TRY_HIP(launch_fill_i32(B.err, 2, 0, s->st));

    // tokens grouped by count row (the count rebuild walks rows); the rows
    // whose (group, word) pair occurs at most kNarrowMax times (fixed by the
    // corpus) also get 16-bit copies
    unsigned long long n_narrow = 0;
    {
        int rc2 = dev_alloc(s, &B.perm, N, "row-sorted tokens");
        if (!assoc) {  // the plain model's rebuild gathers from routed states
            if (rc2 == SPDP_OK) rc2 = dev_alloc(s, &B.tok_slot, N, "state route of tokens");
            if (rc2 == SPDP_OK) rc2 = dev_alloc(s, &B.row_slot, N, "state route of row entries");
            if (rc2 == SPDP_OK) rc2 = dev_alloc(s, &B.zr_b, N, "routed states");
        }
        if (rc2 == SPDP_OK) rc2 = dev_alloc(s, &B.row_off, rows + 1, "row offsets");
        if (rc2 == SPDP_OK) rc2 = dev_alloc(s, &B.row_narrow, rows, "narrow-row flags");
        if (rc2 == SPDP_OK) rc2 = dev_alloc(s, &B.tok_narrow, N, "narrow-row flags of tokens");
        if (rc2 != SPDP_OK) cleanup_staging();
        TRY(rc2);
        e = build_row_index(m, B, gw_count, s->st);
        if (e == hipSuccess) e = launch_fill_u64(B.ctr, 4, 0, s->st);
        if (e == hipSuccess)
            e = launch_narrow_flags(m, B.gw, gw_count, B.row_narrow, B.tok_narrow, B.ctr, s->st);
        if (e == hipSuccess)
            e = hipMemcpyAsync(&n_narrow, B.ctr, sizeof n_narrow, hipMemcpyDeviceToHost, s->st);
        if (e == hipSuccess) e = hipStreamSynchronize(s->st);
        cleanup_staging();
        TRY_HIP(e);
    }
    s->n_narrow_rows = (int64_t)n_narrow;

    // word associations
    if (assoc) TRY(upload_assoc(s, assoc));

    // Stirling cache
    const int64_t n_logS = tri_index(m.ncap + 1, 0);  // rows 0..ncap
    const int64_t n_Q = tri_index(m.ncap, 0);         // rows 0..ncap-1
    if (m.ncap > kMaxNcap || n_logS * 8 + n_Q * 24 > kStirlingBudget)
        TRY(fail(SPDP_E_RANGE,
                 "a (group, word) pair occurs %d times; the Stirling cache covers at most %d",
                 m.ncap, kMaxNcap));
    TRY(dev_alloc(s, &B.logS, n_logS, "log Stirling table"));
    TRY(dev_alloc(s, &B.Q, n_Q, "Stirling ratio pairs"));
    TRY(dev_alloc(s, &B.Q64, n_Q, "fp64 Stirling ratio pairs"));
    TRY(dev_alloc(s, &B.lfact, (int64_t)m.ncap + 1, "log factorials"));
    TRY_HIP(launch_stirling(m, B.logS, B.Q, B.Q64, B.lfact, s->st));

    // state and counts
    TRY(dev_alloc(s, &B.zr[0], N, "zr"));
    TRY(dev_alloc(s, &B.zr[1], N, "zr"));
    TRY(dev_alloc(s, &B.nt, rows * m.Kp, "packed customer/table counts"));
    TRY(dev_alloc(s, &B.B, (int64_t)V * m.Kp, "shadow-base table counts"));
    TRY(dev_alloc(s, &B.B16, (int64_t)V * m.Kp, "16-bit shadow-base table counts"));
    TRY(dev_alloc(s, &B.wide, 1, "shadow-base width flag"));
    TRY_HIP(launch_fill_i32(B.nt, rows * m.Kp, 0, s->st));
    // (the 16-bit copies: a buffer of the full row count, so that row q's copy
    // sits at q Kp; only the narrow rows' copies are written and read; the
    // sampler's vector reads of a narrow row run at most 4 cells past its
    // end, which the 64-cell tail keeps inside the buffer)
    const int64_t n16 = (n_narrow > 0 ? rows * m.Kp : 0) + 64;
    TRY(dev_alloc(s, &B.nt16, n16, "narrow count rows"));
    TRY_HIP(launch_fill_i32(reinterpret_cast<int32_t *>(B.nt16), n16 / 2, 0, s->st));
    TRY(dev_alloc(s, &B.Ngk, (int64_t)G * m.Kp, "N_gk"));
    TRY(dev_alloc(s, &B.Tgk, (int64_t)G * m.Kp, "T_gk"));
    TRY(dev_alloc(s, &B.Bk, m.Kp, "B_k"));
    TRY(dev_alloc(s, &B.f0, (int64_t)G * m.Kp, "f0"));
    TRY(dev_alloc(s, &B.f1, (int64_t)G * m.Kp, "f1"));
    TRY(dev_alloc(s, &B.fk, 3 * (int64_t)G * m.Kp, "removal factors"));
    TRY(dev_alloc(s, &B.rep_part, rows, "repair partial counts"));
    TRY(dev_alloc(s, &B.part, stat_partials_needed(), "reduction partials"));
    {
        TRY(dev_alloc(s, &B.exact, 1, "sampler context"));
        ExactCtx x{};
        x.Ngk = B.Ngk;
        x.Tgk = B.Tgk;
        x.Bk = B.Bk;
        x.B = B.B;
        x.logS = B.logS;
        x.Q64 = B.Q64;
        x.a = a;
        x.b = b;
        x.Vgamma = (double)V * gamma;
        x.alpha = alpha;
        x.gamma = gamma;
        x.K = K;
        x.ncap = m.ncap;
        x.srcrec = B.srcrec;
        x.p64 = B.p64;
        x.Sp = m.Sp;
        TRY_HIP(hipMemcpyAsync(B.exact, &x, sizeof x, hipMemcpyHostToDevice, s->st));
        TRY_HIP(hipStreamSynchronize(s->st));
    }
    B.partial_len = loglik_partials_needed();
    TRY(dev_alloc(s, &B.partial, B.partial_len, "loglik partials"));
    s->cur = 0;
    TRY_HIP(launch_init_z(m, corpus->init_seed, B.zr[0], s->st));
    TRY(rebuild_state(s));
    TRY(sync(s));
#undef TRY
#undef TRY_HIP
    *out = s;
    return SPDP_OK;
}

}  // namespace

extern "C" {

void spdp_destroy(spdp_state *s) { free_state(s); }

int spdp_sweep(spdp_state *s, uint32_t sweep, uint64_t seed)
{
    if (!s) return fail(SPDP_E_ARG, "state is NULL");
    HIP_TRY(hipSetDevice(s->device));
    const Model &m = s->m;
    DeviceBuffers &b = s->b;
    int32_t *zr_old = b.zr[s->cur], *zr_new = b.zr[1 - s->cur];
    int rc;
    if ((rc = timed(s, 3, [&] { return launch_factors(m, b, s->st); })) != SPDP_OK) return rc;
    if (m.Sp > 0) {
        // word associations: source-keyed shadow base, rebuilt by the row pass
        if ((rc = timed(s, 0, [&] {
                 return launch_sample_assoc(m, b, zr_old, zr_new, sweep, seed, nullptr, nullptr,
                                            0, 0, s->st);
             })) != SPDP_OK)
            return rc;
        if ((rc = timed(s, 1, [&] { return launch_rows_assoc(m, b, zr_new, s->st); })) != SPDP_OK)
            return rc;
        if ((rc = timed(s, 2, [&] { return launch_base16(m, b, s->st); })) != SPDP_OK) return rc;
    } else {
        if ((rc = timed(s, 0, [&] {
                 return launch_sample(m, b, zr_old, zr_new, sweep, seed, nullptr, nullptr, 0, 0,
                                      s->st);
             })) != SPDP_OK)
            return rc;
        if ((rc = timed(s, 1, [&] { return launch_rows(m, b, zr_new, s->st); })) != SPDP_OK)
            return rc;
        if ((rc = timed(s, 2, [&] { return launch_base16(m, b, s->st); })) != SPDP_OK) return rc;
    }
    s->rows32 = false;
    if ((rc = timed(s, 3, [&] { return launch_totals(m, b, zr_new, s->st); })) != SPDP_OK) return rc;
    s->cur = 1 - s->cur;
    return SPDP_OK;
}

int spdp_sweep_async(spdp_state *s, uint32_t sweep, uint64_t seed, int32_t waves,
                     int32_t live_totals)
{
    if (!s) return fail(SPDP_E_ARG, "state is NULL");
    const Model &m = s->m;
    if (m.Sp > 0) return fail(SPDP_E_ARG, "the asynchronous sweep is built for P = I only");
    if (waves < 0) return fail(SPDP_E_ARG, "waves must be >= 0");
    HIP_TRY(hipSetDevice(s->device));
    DeviceBuffers &b = s->b;
    int rc;
    if (!b.order) {
        if ((rc = dev_alloc(s, &b.order, m.N, "visiting order")) != SPDP_OK) return rc;
        if ((rc = dev_alloc(s, &b.tok_doc, m.N, "token documents")) != SPDP_OK) return rc;
        if ((rc = dev_alloc(s, &b.cdk, (int64_t)m.D * m.Kp, "document counts")) != SPDP_OK)
            return rc;
        HIP_TRY(build_visit_order(m, b, s->st));
    }
    if (waves == 0) {
        int cus = 0;
        HIP_TRY(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, s->device));
        waves = 16 * (cus > 0 ? cus : 1);
    }
    // the pass updates the state in place, in the other buffer, so that the
    // statistics compare it with the state before the sweep
    int32_t *zr_old = b.zr[s->cur], *zr_new = b.zr[1 - s->cur];
    if (m.N > 0)
        HIP_TRY(hipMemcpyAsync(zr_new, zr_old, (size_t)m.N * sizeof(int32_t),
                               hipMemcpyDeviceToDevice, s->st));
    // the pass reads and updates the 32-bit rows of every row
    HIP_TRY(widen_rows(s));
    if ((rc = timed(s, 3, [&] { return launch_doc_counts(m, b, zr_new, b.cdk, s->st); })) != SPDP_OK)
        return rc;
    if ((rc = timed(s, 0, [&] {
             return launch_sample_async(m, b, b.order, b.tok_doc, b.cdk, zr_new, sweep, seed,
                                        waves, live_totals != 0, s->st);
         })) != SPDP_OK)
        return rc;
    if ((rc = timed(s, 1, [&] { return launch_rows(m, b, zr_new, s->st); })) != SPDP_OK) return rc;
    if ((rc = timed(s, 2, [&] { return launch_base16(m, b, s->st); })) != SPDP_OK) return rc;
    s->rows32 = false;
    if ((rc = timed(s, 3, [&] { return launch_totals(m, b, zr_new, s->st); })) != SPDP_OK) return rc;
    s->cur = 1 - s->cur;
    return SPDP_OK;
}

int spdp_counts(const spdp_state *s, int32_t g_begin, int32_t g_end, int32_t *n_gkw,
                int32_t *t_gkw, int where)
{
    if (!s) return fail(SPDP_E_ARG, "state is NULL");
    const Model &m = s->m;
    if (g_begin < 0 || g_end > m.G || g_begin > g_end) return fail(SPDP_E_ARG, "bad group range");
    if (where != 0 && where != 1) return fail(SPDP_E_ARG, "where must be 0 or 1");
    HIP_TRY(hipSetDevice(s->device));
    if (!n_gkw && !t_gkw) return SPDP_OK;
    HIP_TRY(widen_rows(s));
    const int64_t cells = (int64_t)m.V * m.K;
    int32_t *stage_n = nullptr, *stage_t = nullptr;
    if (where == 0) {
        // one group at a time through device staging buffers
        HIP_TRY(hipMalloc(&stage_n, (size_t)cells * 4));
        hipError_t e = hipMalloc(&stage_t, (size_t)cells * 4);
        if (e != hipSuccess) {
            (void)hipFree(stage_n);
            HIP_TRY(e);
        }
    }
    hipError_t e = hipSuccess;
    for (int32_t g = g_begin; g < g_end && e == hipSuccess; ++g) {
        const int64_t off = (int64_t)(g - g_begin) * cells;
        if (where == 1) {
            e = launch_unpack_counts(m, s->b, g, n_gkw ? n_gkw + off : nullptr,
                                     t_gkw ? t_gkw + off : nullptr, s->st);
        } else {
            e = launch_unpack_counts(m, s->b, g, stage_n, stage_t, s->st);
            if (e == hipSuccess && n_gkw)
                e = hipMemcpyAsync(n_gkw + off, stage_n, (size_t)cells * 4, hipMemcpyDeviceToHost, s->st);
            if (e == hipSuccess && t_gkw)
                e = hipMemcpyAsync(t_gkw + off, stage_t, (size_t)cells * 4, hipMemcpyDeviceToHost, s->st);
            if (e == hipSuccess) e = hipStreamSynchronize(s->st);
        }
    }
    if (stage_n) (void)hipFree(stage_n);
    if (stage_t) (void)hipFree(stage_t);
    HIP_TRY(e);
    return sync(s);
}

int spdp_totals(const spdp_state *s, int32_t *N_gk, int32_t *T_gk, int32_t *B_wk, int32_t *B_k,
                int where)
{
    if (!s) return fail(SPDP_E_ARG, "state is NULL");
    if (where != 0 && where != 1) return fail(SPDP_E_ARG, "where must be 0 or 1");
    HIP_TRY(hipSetDevice(s->device));
    const Model &m = s->m;
    const hipMemcpyKind kind = where ? hipMemcpyDeviceToDevice : hipMemcpyDeviceToHost;
    const size_t w = (size_t)m.K * 4, p = (size_t)m.Kp * 4;
    if (N_gk) HIP_TRY(hipMemcpy2DAsync(N_gk, w, s->b.Ngk, p, w, (size_t)m.G, kind, s->st));
    if (T_gk) HIP_TRY(hipMemcpy2DAsync(T_gk, w, s->b.Tgk, p, w, (size_t)m.G, kind, s->st));
    if (B_wk) HIP_TRY(hipMemcpy2DAsync(B_wk, w, s->b.B, p, w, (size_t)m.V, kind, s->st));
    if (B_k) HIP_TRY(hipMemcpyAsync(B_k, s->b.Bk, w, kind, s->st));
    return sync(s);
}

int spdp_loglik(spdp_state *s, double *out)
{
    if (!s || !out) return fail(SPDP_E_ARG, "null argument");
    HIP_TRY(hipSetDevice(s->device));
    HIP_TRY(widen_rows(s));
    HIP_TRY(launch_fill_i32(s->b.err, 2, 0, s->st));
    HIP_TRY(launch_loglik(s->m, s->b, s->b.zr[s->cur], s->st));
    double v = 0.0;
    HIP_TRY(hipMemcpyAsync(&v, s->b.scalar, sizeof v, hipMemcpyDeviceToHost, s->st));
    int32_t herr[2];
    int rc = check_device_flags(s, herr);
    if (rc != SPDP_OK) return rc;
    if (herr[0]) return fail(SPDP_E_STATE, "count state has a cell with t > n or t = 0 < n");
    *out = v;
    return SPDP_OK;
}

int spdp_estimates(spdp_state *s, int32_t g_begin, int32_t g_end, double *theta, double *phi0,
                   double *phi, int where)
{
    if (!s) return fail(SPDP_E_ARG, "state is NULL");
    const Model &m = s->m;
    if (where != 0 && where != 1) return fail(SPDP_E_ARG, "where must be 0 or 1");
    if (phi && (g_begin < 0 || g_end > m.G || g_begin > g_end))
        return fail(SPDP_E_ARG, "bad group range");
    HIP_TRY(hipSetDevice(s->device));
    if (phi) HIP_TRY(widen_rows(s));
    const int64_t vk = (int64_t)m.V * m.K, dk = (int64_t)m.D * m.K;
    // device destinations (the caller's buffers, or one staging buffer reused)
    double *stage = nullptr;
    if (where == 0) {
        int64_t need = 0;
        if (theta) need = dk;
        if ((phi0 || phi) && vk > need) need = vk;
        if (need > 0) HIP_TRY(hipMalloc(&stage, (size_t)need * sizeof(double)));
    }
    hipError_t e = hipSuccess;
    auto out = [&](double *dst, int64_t n, auto &&launch) {
        if (e != hipSuccess || !dst || n <= 0) return;
        e = launch(where ? dst : stage);
        if (e == hipSuccess && where == 0)
            e = hipMemcpyAsync(dst, stage, (size_t)n * sizeof(double), hipMemcpyDeviceToHost,
                               s->st);
        if (e == hipSuccess && where == 0) e = hipStreamSynchronize(s->st);
    };
    out(theta, dk, [&](double *d) { return launch_theta(m, s->b, s->b.zr[s->cur], d, s->st); });
    out(phi0, vk, [&](double *d) { return launch_phi0(m, s->b, d, s->st); });
    for (int32_t g = g_begin; phi && g < g_end; ++g)
        out(phi + (int64_t)(g - g_begin) * vk, vk,
            [&](double *d) { return launch_phig(m, s->b, g, d, s->st); });
    if (stage) (void)hipFree(stage);
    HIP_TRY(e);
    return sync(s);
}

int spdp_heldout(spdp_state *s, const spdp_corpus *test, const spdp_groups *test_groups,
                 int32_t n_sweeps, uint64_t seed, double *out2, int32_t *z_out, int where)
{
    if (!s || !test || !test_groups || !out2) return fail(SPDP_E_ARG, "null argument");
    const Model &m = s->m;
    if (where != 0 && where != 1) return fail(SPDP_E_ARG, "where must be 0 or 1");
    if (n_sweeps < 0) return fail(SPDP_E_ARG, "n_sweeps < 0");
    const int64_t N = test->n_tokens;
    const int32_t D = test->n_docs;
    if (N < 0 || N >= (1ll << 31) || D < 0) return fail(SPDP_E_ARG, "bad test corpus size");
    if (test->vocab != m.V) return fail(SPDP_E_ARG, "test vocabulary differs from the state's");
    if (test_groups->n_groups != m.G) return fail(SPDP_E_ARG, "test groups differ from the state's");
    if ((N > 0 && !test->words) || !test->doc_offsets || (D > 0 && !test_groups->doc_group))
        return fail(SPDP_E_ARG, "null test array");
    if (test->doc_offsets[0] != 0 || test->doc_offsets[D] != N)
        return fail(SPDP_E_ARG, "test doc_offsets must run from 0 to n_tokens");
    std::vector<int32_t> gw((size_t)(N > 0 ? N : 1));
    for (int32_t d = 0; d < D; ++d) {
        const int64_t b0 = test->doc_offsets[d], b1 = test->doc_offsets[d + 1];
        const int32_t g = test_groups->doc_group[d];
        if (b1 < b0) return fail(SPDP_E_ARG, "test doc_offsets decrease");
        if (g < 0 || g >= m.G) return fail(SPDP_E_ARG, "test doc_group out of [0, n_groups)");
        for (int64_t i = b0; i < b1; ++i) {
            const int32_t w = test->words[i];
            if (w < 0 || w >= m.V) return fail(SPDP_E_ARG, "test word id out of [0, vocab)");
            gw[(size_t)i] = g * m.V + w;
        }
    }
    HIP_TRY(hipSetDevice(s->device));
    HIP_TRY(widen_rows(s));
    int32_t *gw_d = nullptr, *grp_d = nullptr, *z_d = nullptr;
    int64_t *off_d = nullptr;
    double *ll_d = nullptr;
    hipError_t e = hipMalloc(&gw_d, (size_t)(N > 0 ? N : 1) * 4);
    if (e == hipSuccess) e = hipMalloc(&z_d, (size_t)(N > 0 ? N : 1) * 4);
    if (e == hipSuccess) e = hipMalloc(&off_d, (size_t)(D + 1) * 8);
    if (e == hipSuccess) e = hipMalloc(&grp_d, (size_t)(D > 0 ? D : 1) * 4);
    if (e == hipSuccess) e = hipMalloc(&ll_d, (size_t)(D > 0 ? D : 1) * 8);
    if (e == hipSuccess && N > 0)
        e = hipMemcpyAsync(gw_d, gw.data(), (size_t)N * 4, hipMemcpyHostToDevice, s->st);
    if (e == hipSuccess)
        e = hipMemcpyAsync(off_d, test->doc_offsets, (size_t)(D + 1) * 8, hipMemcpyHostToDevice,
                           s->st);
    if (e == hipSuccess && D > 0)
        e = hipMemcpyAsync(grp_d, test_groups->doc_group, (size_t)D * 4, hipMemcpyHostToDevice,
                           s->st);
    if (e == hipSuccess)
        e = launch_foldin(m, s->b, D, gw_d, off_d, grp_d, n_sweeps, seed, z_d, ll_d, s->st);
    std::vector<double> ll((size_t)(D > 0 ? D : 1), 0.0);
    if (e == hipSuccess && D > 0)
        e = hipMemcpyAsync(ll.data(), ll_d, (size_t)D * 8, hipMemcpyDeviceToHost, s->st);
    if (e == hipSuccess && z_out && N > 0)
        e = hipMemcpyAsync(z_out, z_d, (size_t)N * 4,
                           where ? hipMemcpyDeviceToDevice : hipMemcpyDeviceToHost, s->st);
    if (e == hipSuccess) e = hipStreamSynchronize(s->st);
    (void)hipFree(gw_d);
    (void)hipFree(z_d);
    (void)hipFree(off_d);
    (void)hipFree(grp_d);
    (void)hipFree(ll_d);
    HIP_TRY(e);
    double total = 0.0;  // documents in order
    for (int32_t d = 0; d < D; ++d) total += ll[(size_t)d];
    out2[0] = N > 0 ? exp(-total / (double)N) : NAN;
    out2[1] = total;
    return SPDP_OK;
}

int spdp_hellinger(spdp_state *s, const double *p, int32_t kp, const double *q, int32_t kq,
                   int32_t n_outcomes, double *h, int where)
{
    if (!s || !q || !h) return fail(SPDP_E_ARG, "null argument");
    const Model &m = s->m;
    if (where != 0 && where != 1) return fail(SPDP_E_ARG, "where must be 0 or 1");
    if (kp < 0 || kq < 0 || n_outcomes < 0) return fail(SPDP_E_ARG, "negative size");
    if (kp > SPDP_MAX_K || kq > SPDP_MAX_K)
        return fail(SPDP_E_ARG, "topic counts must be at most %d", SPDP_MAX_K);
    if (!p && (kp != m.K || n_outcomes != m.V))
        return fail(SPDP_E_ARG, "with p NULL (the state's phi0), kp must be K and n_outcomes V");
    HIP_TRY(hipSetDevice(s->device));
    const int64_t V = n_outcomes, np = V * kp, nq = V * kq, nh = (int64_t)kp * kq;
    const HellingerPlan plan = hellinger_plan(kp, kq, V);
    std::vector<void *> tmp;
    hipError_t e = hipSuccess;
    auto dalloc = [&](int64_t n) -> double * {
        void *x = nullptr;
        if (e == hipSuccess) e = hipMalloc(&x, (size_t)(n > 0 ? n : 1) * sizeof(double));
        if (e != hipSuccess) return nullptr;
        tmp.push_back(x);
        return (double *)x;
    };
    auto upload = [&](const double *src, int64_t n) -> const double * {
        double *x = dalloc(n);
        if (e == hipSuccess && n > 0)
            e = hipMemcpyAsync(x, src, (size_t)n * sizeof(double), hipMemcpyHostToDevice, s->st);
        return x;
    };
    const double *Pd = p, *Qd = q;
    double *Hd = h;
    if (!p) {
        double *x = dalloc(np);
        if (e == hipSuccess) e = launch_phi0(m, s->b, x, s->st);
        Pd = x;
    } else if (!where) {
        Pd = upload(p, np);
    }
    if (!where) {
        Qd = upload(q, nq);
        Hd = dalloc(nh);
    }
    double *part = dalloc((int64_t)plan.slices * nh);
    if (e == hipSuccess) e = launch_hellinger(plan, Pd, kp, Qd, kq, V, part, Hd, s->st);
    if (e == hipSuccess && !where && nh > 0)
        e = hipMemcpyAsync(h, Hd, (size_t)nh * sizeof(double), hipMemcpyDeviceToHost, s->st);
    if (e == hipSuccess) e = hipStreamSynchronize(s->st);
    for (void *x : tmp) (void)hipFree(x);
    HIP_TRY(e);
    return SPDP_OK;
}

int spdp_hellinger_noalloc(spdp_state *s, const double *p, int32_t kp, const double *q,
                           int32_t kq, int32_t n_outcomes, double *h)
{
    if (!s || !p || !q || !h) return fail(SPDP_E_ARG, "null argument");
    if (kp < 0 || kq < 0 || n_outcomes < 0) return fail(SPDP_E_ARG, "negative size");
    if (kp > SPDP_MAX_K || kq > SPDP_MAX_K)
        return fail(SPDP_E_ARG, "topic counts must be at most %d", SPDP_MAX_K);
    const int64_t nh = (int64_t)kp * kq;
    if (nh > kHellingerScratch)
        return fail(SPDP_E_RANGE, "kp * kq = %lld exceeds the %lld partial sums of the static "
                    "scratch", (long long)nh, (long long)kHellingerScratch);
    HIP_TRY(hipSetDevice(s->device));
    double *part = nullptr;
    HIP_TRY((hipError_t)hellinger_scratch(s->device, &part));
    // p, q and h must be device memory holding their sizes (the kernels read
    // and write them directly)
    const struct {
        const void *ptr;
        int64_t bytes;
        const char *name;
    } bufs[3] = {{p, (int64_t)n_outcomes * kp * 8, "p"},
                 {q, (int64_t)n_outcomes * kq * 8, "q"},
                 {h, nh * 8, "h"}};
    for (const auto &x : bufs) {
        hipDeviceptr_t base = nullptr;
        size_t size = 0;
        if (hipMemGetAddressRange(&base, &size, const_cast<void *>(x.ptr)) != hipSuccess) {
            (void)hipGetLastError();
            return fail(SPDP_E_ARG, "%s is not device memory", x.name);
        }
        if (static_cast<const char *>(x.ptr) + x.bytes > static_cast<const char *>(base) + size)
            return fail(SPDP_E_ARG, "%s: %lld bytes run past its allocation", x.name,
                        (long long)x.bytes);
    }
    const HellingerPlan plan = hellinger_plan(kp, kq, n_outcomes, kHellingerScratch);
    HIP_TRY(launch_hellinger(plan, p, kp, q, kq, n_outcomes, part, h, s->st));
    return SPDP_OK;
}

int spdp_align_topics(const double *h, int32_t kp, int32_t kq, int32_t *match, double *total)
{
    if (!total || (kp > 0 && (!h || !match))) return fail(SPDP_E_ARG, "null argument");
    if (kp < 0 || kq < kp) return fail(SPDP_E_ARG, "need 0 <= kp <= kq");
    for (int64_t i = 0; i < (int64_t)kp * kq; ++i)
        if (!std::isfinite(h[i])) return fail(SPDP_E_ARG, "distance matrix entry is not finite");
    *total = kp > 0 ? align_topics_host(h, kp, kq, match) : 0.0;
    return SPDP_OK;
}

int spdp_get_assignments(const spdp_state *s, int32_t *z, uint8_t *r, int where)
{
    if (!s) return fail(SPDP_E_ARG, "state is NULL");
    if (where != 0 && where != 1) return fail(SPDP_E_ARG, "where must be 0 or 1");
    HIP_TRY(hipSetDevice(s->device));
    const Model &m = s->m;
    if (m.N == 0 || (!z && !r)) return SPDP_OK;
    if (where == 1) {
        HIP_TRY(launch_unpack_zr(m, s->b.zr[s->cur], z, r, s->st));
        return sync(s);
    }
    int32_t *zd = nullptr;
    uint8_t *rd = nullptr;
    HIP_TRY(hipMalloc(&zd, (size_t)m.N * sizeof(int32_t)));
    hipError_t e = hipMalloc(&rd, (size_t)m.N);
    if (e == hipSuccess) e = launch_unpack_zr(m, s->b.zr[s->cur], zd, rd, s->st);
    if (e == hipSuccess && z) e = hipMemcpyAsync(z, zd, (size_t)m.N * 4, hipMemcpyDeviceToHost, s->st);
    if (e == hipSuccess && r) e = hipMemcpyAsync(r, rd, (size_t)m.N, hipMemcpyDeviceToHost, s->st);
    if (e == hipSuccess) e = hipStreamSynchronize(s->st);
    (void)hipFree(zd);
    if (rd) (void)hipFree(rd);
    HIP_TRY(e);
    return SPDP_OK;
}

}  // extern "C"

namespace {

// Replace the state by (z, r[, s]) and rebuild; slots only with associations.
int set_state(spdp_state *s, const int32_t *z, const uint8_t *r, const uint8_t *sl, int where)
{
    if (where != 0 && where != 1) return fail(SPDP_E_ARG, "where must be 0 or 1");
    HIP_TRY(hipSetDevice(s->device));
    const Model &m = s->m;
    if (m.N > 0) {
        const int32_t *zd = z;
        const uint8_t *rd = r, *sd = sl;
        int32_t *zt = nullptr;
        uint8_t *rt = nullptr, *st8 = nullptr;
        auto release = [&]() {
            if (zt) (void)hipFree(zt);
            if (rt) (void)hipFree(rt);
            if (st8) (void)hipFree(st8);
        };
        if (where == 0) {
            hipError_t e = hipMalloc(&zt, (size_t)m.N * sizeof(int32_t));
            if (e == hipSuccess) e = hipMalloc(&rt, (size_t)m.N);
            if (e == hipSuccess && sl) e = hipMalloc(&st8, (size_t)m.N);
            if (e == hipSuccess)
                e = hipMemcpyAsync(zt, z, (size_t)m.N * 4, hipMemcpyHostToDevice, s->st);
            if (e == hipSuccess) e = hipMemcpyAsync(rt, r, (size_t)m.N, hipMemcpyHostToDevice, s->st);
            if (e == hipSuccess && sl)
                e = hipMemcpyAsync(st8, sl, (size_t)m.N, hipMemcpyHostToDevice, s->st);
            if (e != hipSuccess) {
                release();
                HIP_TRY(e);
            }
            zd = zt;
            rd = rt;
            sd = st8;
        }
        HIP_TRY(launch_fill_i32(s->b.err, 2, 0, s->st));
        hipError_t e = m.Sp > 0 ? launch_pack_zrs(m, s->b, zd, rd, sd, s->b.zr[s->cur], s->b.err, s->st)
                                : launch_pack_zr(m, zd, rd, s->b.zr[s->cur], s->b.err, s->st);
        int32_t herr[2] = {0, 0};
        if (e == hipSuccess) e = hipMemcpyAsync(herr, s->b.err, sizeof herr, hipMemcpyDeviceToHost, s->st);
        if (e == hipSuccess) e = hipStreamSynchronize(s->st);
        release();
        HIP_TRY(e);
        if (herr[0] & 4)
            return fail(SPDP_E_ARG, m.Sp > 0 ? "z out of [0, K), r not in {0, 1}, or a head's "
                                               "slot is not a source of its row"
                                             : "z out of [0, K) or r not in {0, 1}");
    }
    int rc = rebuild_state(s);
    if (rc != SPDP_OK) return rc;
    return sync(s);
}

}  // namespace

extern "C" {

int spdp_set_assignments(spdp_state *s, const int32_t *z, const uint8_t *r, int where)
{
    if (!s || !z || !r) return fail(SPDP_E_ARG, "null argument");
    return set_state(s, z, r, nullptr, where);
}

int spdp_set_assignments_assoc(spdp_state *s, const int32_t *z, const uint8_t *r,
                               const uint8_t *slot, int where)
{
    if (!s || !z || !r || !slot) return fail(SPDP_E_ARG, "null argument");
    if (s->m.Sp == 0) return fail(SPDP_E_ARG, "the state has no word associations");
    return set_state(s, z, r, slot, where);
}

int spdp_get_slots(const spdp_state *s, uint8_t *slot, int where)
{
    if (!s || !slot) return fail(SPDP_E_ARG, "null argument");
    if (where != 0 && where != 1) return fail(SPDP_E_ARG, "where must be 0 or 1");
    HIP_TRY(hipSetDevice(s->device));
    const Model &m = s->m;
    if (m.N == 0) return SPDP_OK;
    if (where == 1) {
        HIP_TRY(launch_unpack_slot(m, s->b.zr[s->cur], slot, s->st));
        return sync(s);
    }
    uint8_t *sd = nullptr;
    HIP_TRY(hipMalloc(&sd, (size_t)m.N));
    hipError_t e = launch_unpack_slot(m, s->b.zr[s->cur], sd, s->st);
    if (e == hipSuccess) e = hipMemcpyAsync(slot, sd, (size_t)m.N, hipMemcpyDeviceToHost, s->st);
    if (e == hipSuccess) e = hipStreamSynchronize(s->st);
    (void)hipFree(sd);
    HIP_TRY(e);
    return SPDP_OK;
}

int spdp_max_sources(const spdp_state *s, int32_t *S)
{
    if (!s || !S) return fail(SPDP_E_ARG, "null argument");
    *S = s->m.S;
    return SPDP_OK;
}

int spdp_debug_conditionals(spdp_state *s, uint32_t sweep, uint64_t seed, int64_t tok_begin,
                            int64_t tok_end, float *w_out, float *u_out, int32_t *zr_out,
                            int where)
{
    if (!s) return fail(SPDP_E_ARG, "state is NULL");
    const Model &m = s->m;
    if (tok_begin < 0 || tok_end > m.N || tok_begin > tok_end)
        return fail(SPDP_E_ARG, "bad token range");
    if (where != 0 && where != 1) return fail(SPDP_E_ARG, "where must be 0 or 1");
    HIP_TRY(hipSetDevice(s->device));
    DeviceBuffers &b = s->b;
    const int64_t T = tok_end - tok_begin;
    if (T == 0) return SPDP_OK;
    // outcomes per token: 2K, or K (S + 1) with word associations
    const int64_t nout = m.Sp > 0 ? (int64_t)m.K * (m.S + 1) : 2 * (int64_t)m.K;
    if (!b.zr_dbg) {
        void *p = nullptr;
        if (hipMalloc(&p, (size_t)m.N * sizeof(int32_t)) != hipSuccess) {
            (void)hipGetLastError();
            return fail(SPDP_E_NOMEM, "debug state buffer");
        }
        b.zr_dbg = (int32_t *)p;
    }
    const bool trace = (w_out != nullptr || u_out != nullptr);
    if (trace && T > b.tr_cap) {
        if (b.tr_w) (void)hipFree(b.tr_w);
        if (b.tr_u) (void)hipFree(b.tr_u);
        b.tr_w = nullptr;
        b.tr_u = nullptr;
        b.tr_cap = 0;
        void *p = nullptr;
        if (hipMalloc(&p, (size_t)(T * nout) * sizeof(float)) != hipSuccess) {
            (void)hipGetLastError();
            return fail(SPDP_E_NOMEM, "trace buffer");
        }
        b.tr_w = (float *)p;
        if (hipMalloc(&p, (size_t)T * sizeof(float)) != hipSuccess) {
            (void)hipGetLastError();
            return fail(SPDP_E_NOMEM, "trace buffer");
        }
        b.tr_u = (float *)p;
        b.tr_cap = T;
    }
    if (trace) {
        HIP_TRY(launch_fill_i32((int32_t *)b.tr_w, T * nout, 0, s->st));
        HIP_TRY(launch_fill_i32((int32_t *)b.tr_u, T, 0, s->st));
    }
    int32_t *zr_old = b.zr[s->cur], *zr_tmp = b.zr_dbg;
    HIP_TRY(launch_factors(m, b, s->st));
    if (m.Sp > 0)
        HIP_TRY(launch_sample_assoc(m, b, zr_old, zr_tmp, sweep, seed, trace ? b.tr_w : nullptr,
                                    trace ? b.tr_u : nullptr, tok_begin, tok_end, s->st));
    else
        HIP_TRY(launch_sample(m, b, zr_old, zr_tmp, sweep, seed, trace ? b.tr_w : nullptr,
                              trace ? b.tr_u : nullptr, tok_begin, tok_end, s->st));
    const hipMemcpyKind kind = where ? hipMemcpyDeviceToDevice : hipMemcpyDeviceToHost;
    if (w_out) HIP_TRY(hipMemcpyAsync(w_out, b.tr_w, (size_t)(T * nout) * 4, kind, s->st));
    if (u_out) HIP_TRY(hipMemcpyAsync(u_out, b.tr_u, (size_t)T * 4, kind, s->st));
    if (zr_out) HIP_TRY(hipMemcpyAsync(zr_out, zr_tmp + tok_begin, (size_t)T * 4, kind, s->st));
    return sync(s);
}

int spdp_stats(const spdp_state *s, int64_t *changed, int64_t *repaired)
{
    if (!s) return fail(SPDP_E_ARG, "state is NULL");
    HIP_TRY(hipSetDevice(s->device));
    unsigned long long c[4];
    HIP_TRY(launch_stat_sums(s->m, s->b, s->b.zr[s->cur], s->b.zr[1 - s->cur], s->st));
    HIP_TRY(hipMemcpyAsync(c, s->b.ctr, sizeof c, hipMemcpyDeviceToHost, s->st));
    int rc = sync(s);
    if (rc != SPDP_OK) return rc;
    if (changed) *changed = (int64_t)c[0];
    if (repaired) *repaired = (int64_t)c[1];
    return SPDP_OK;
}

int spdp_read_probe(const void *buf, int64_t bytes, int32_t row_bytes, int64_t rows,
                    int32_t waves, void *stream, double *ms)
{
    if (!buf || !ms) return fail(SPDP_E_ARG, "buf or ms is NULL");
    if ((reinterpret_cast<uintptr_t>(buf) & 15) != 0)
        return fail(SPDP_E_ARG, "buf is not 16-byte aligned");
    if (!(row_bytes == 0 || row_bytes == 1024 || row_bytes == 2048 || row_bytes == 3072 ||
          row_bytes == 4096 || row_bytes == 8192))
        return fail(SPDP_E_ARG, "row_bytes %d is not 0, 1024, 2048, 3072, 4096 or 8192",
                    row_bytes);
    if (bytes < 16 || (row_bytes > 0 && bytes < row_bytes))
        return fail(SPDP_E_ARG, "bytes %lld is below one row", (long long)bytes);
    if (waves < 1 || waves > (1 << 20)) return fail(SPDP_E_ARG, "waves %d not in [1, 2^20]", waves);
    if (row_bytes > 0 && rows < 1) return fail(SPDP_E_ARG, "rows must be positive");
    hipDeviceptr_t base = nullptr;
    size_t size = 0;
    if (hipMemGetAddressRange(&base, &size, const_cast<void *>(buf)) != hipSuccess) {
        (void)hipGetLastError();
        return fail(SPDP_E_ARG, "buf is not device memory");
    }
    const char *b0 = static_cast<const char *>(base);
    if (static_cast<const char *>(buf) + bytes > b0 + size)
        return fail(SPDP_E_ARG, "bytes %lld run past the allocation", (long long)bytes);
    hipStream_t st = static_cast<hipStream_t>(stream);
    hipEvent_t a = nullptr, b = nullptr;
    hipError_t e = hipEventCreate(&a);
    if (e == hipSuccess) e = hipEventCreate(&b);
    if (e == hipSuccess) e = hipEventRecord(a, st);
    if (e == hipSuccess) e = launch_read_probe(buf, bytes, row_bytes, rows, waves, st);
    if (e == hipSuccess) e = hipEventRecord(b, st);
    if (e == hipSuccess) e = hipEventSynchronize(b);
    float t = 0.0f;
    if (e == hipSuccess) e = hipEventElapsedTime(&t, a, b);
    if (a) (void)hipEventDestroy(a);
    if (b) (void)hipEventDestroy(b);
    HIP_TRY(e);
    *ms = t;
    return SPDP_OK;
}

int spdp_kernel_timing(spdp_state *s, int enable)
{
    if (!s) return fail(SPDP_E_ARG, "state is NULL");
    HIP_TRY(hipSetDevice(s->device));
    int rc = sync(s);
    if (rc != SPDP_OK) return rc;
    for (auto &v : s->events) {
        for (auto &ev : v) {
            (void)hipEventDestroy(ev.a);
            (void)hipEventDestroy(ev.b);
        }
        v.clear();
    }
    s->timing = enable != 0;
    return SPDP_OK;
}

int spdp_kernel_times(spdp_state *s, double *ms, int64_t *launches)
{
    if (!s) return fail(SPDP_E_ARG, "state is NULL");
    HIP_TRY(hipSetDevice(s->device));
    int rc = sync(s);
    if (rc != SPDP_OK) return rc;
    for (int c = 0; c < SPDP_NKERNELS; ++c) {
        double acc = 0.0;
        for (auto &ev : s->events[c]) {
            float x = 0.0f;
            HIP_TRY(hipEventElapsedTime(&x, ev.a, ev.b));
            acc += x;
        }
        if (ms) ms[c] = acc;
        if (launches) launches[c] = (int64_t)s->events[c].size();
    }
    return SPDP_OK;
}

int spdp_check(spdp_state *s, int64_t *bad)
{
    if (!s) return fail(SPDP_E_ARG, "state is NULL");
    HIP_TRY(hipSetDevice(s->device));
    const Model &m = s->m;
    const int64_t need = 2 * (int64_t)m.G * m.Kp + m.Kp + (m.Sp > 0 ? (int64_t)m.V * m.Kp : 0);
    int32_t *scratch = nullptr;
    if (hipMalloc(&scratch, (size_t)need * sizeof(int32_t)) != hipSuccess) {
        (void)hipGetLastError();
        return fail(SPDP_E_NOMEM, "check scratch of %lld ints", (long long)need);
    }
    unsigned long long c[4] = {0, 0, 0, 0};
    hipError_t e = launch_fill_u64(s->b.ctr, 4, 0, s->st);
    if (e == hipSuccess) e = launch_check(m, s->b, s->b.zr[s->cur], scratch, s->b.ctr, s->st);
    if (e == hipSuccess) e = hipMemcpyAsync(c, s->b.ctr, sizeof c, hipMemcpyDeviceToHost, s->st);
    if (e == hipSuccess) e = hipStreamSynchronize(s->st);
    (void)hipFree(scratch);
    HIP_TRY(e);
    if (bad) *bad = (int64_t)(c[0] + c[1]);
    if (c[0] || c[1])
        return fail(SPDP_E_STATE,
                    "count state inconsistent: %llu count cells or token states differ from a "
                    "recount of (z, r) or are invalid; %llu totals or shadow-base cells differ",
                    c[0], c[1]);
    return SPDP_OK;
}

int spdp_debug_poke(spdp_state *s, int32_t g, int32_t w, int32_t k, int32_t dn, int32_t dt)
{
    if (!s) return fail(SPDP_E_ARG, "state is NULL");
    const Model &m = s->m;
    if (g < 0 || g >= m.G || w < 0 || w >= m.V || k < 0 || k >= m.K)
        return fail(SPDP_E_ARG, "cell (%d, %d, %d) out of range", g, w, k);
    HIP_TRY(hipSetDevice(s->device));
    // the copy the samplers read: the 16-bit one of a narrow row
    const int64_t q = (int64_t)g * m.V + w;
    uint8_t nar = 0;
    HIP_TRY(hipMemcpyAsync(&nar, s->b.row_narrow + q, 1, hipMemcpyDeviceToHost, s->st));
    int rc = sync(s);
    if (rc != SPDP_OK) return rc;
    const int32_t cap = nar ? kNarrowMax : kCountMax;
    int32_t x = 0;
    if (nar) {
        uint16_t y = 0;
        HIP_TRY(hipMemcpyAsync(&y, s->b.nt16 + q * m.Kp + k, sizeof y, hipMemcpyDeviceToHost, s->st));
        if ((rc = sync(s)) != SPDP_OK) return rc;
        x = wide_of(y);
    } else {
        HIP_TRY(hipMemcpyAsync(&x, s->b.nt + q * m.Kp + k, sizeof x, hipMemcpyDeviceToHost, s->st));
        if ((rc = sync(s)) != SPDP_OK) return rc;
    }
    const int32_t n = (x & kCountMax) + dn, t = (x >> kCountBits) + dt;
    if (n < 0 || n > cap || t < 0 || t > cap)
        return fail(SPDP_E_ARG, "poked counts (%d, %d) out of [0, %d]", n, t, cap);
    x = n | (t << kCountBits);
    if (nar) {
        const uint16_t y = narrow_of(x);
        HIP_TRY(hipMemcpyAsync(s->b.nt16 + q * m.Kp + k, &y, sizeof y, hipMemcpyHostToDevice, s->st));
        s->rows32 = false;
    } else {
        HIP_TRY(hipMemcpyAsync(s->b.nt + q * m.Kp + k, &x, sizeof x, hipMemcpyHostToDevice, s->st));
    }
    return sync(s);
}

int spdp_info(const spdp_state *s, int64_t *out8)
{
    if (!s || !out8) return fail(SPDP_E_ARG, "null argument");
    const Model &m = s->m;
    out8[0] = m.N;
    out8[1] = m.D;
    out8[2] = m.V;
    out8[3] = m.G;
    out8[4] = m.K;
    out8[5] = m.Kp;
    out8[6] = m.ncap;
    out8[7] = s->bytes;
    return SPDP_OK;
}

}  // extern "C"
