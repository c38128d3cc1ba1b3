// hellinger.hip -- Hellinger distances between two topic models (gfx950).
//
// The thesis compares topic models by the Hellinger distance between every
// pair of their topics, the second model's topics re-ordered to line up with
// the first's (chapter "Experiments", subsection "Hellinger Distance").  For
// distributions p, q over the same V outcomes
//   H(p, q)^2 = 1/2 sum_v (sqrt p_v - sqrt q_v)^2 = 1 - BC(p, q),
//   BC(p, q)  = sum_v sqrt(p_v) sqrt(q_v)      (Bhattacharyya coefficient),
// so all kp x kq coefficients are one dense contraction over the outcomes,
//   BC = sqrt(P)^T sqrt(Q),   P [V][kp], Q [V][kq]  (topics contiguous),
// which runs on the fp64 matrix cores: v_mfma_f64_16x16x4 blocks, 64 x 64
// output tiles per 256-thread block, 16 outcomes staged per step through LDS
// with the square roots taken once per staged value.  The outcome axis is
// split into slices so that the grid fills the chip even for small K; the
// slices' partial sums are added in slice order (deterministic) and
// H = sqrt(max(0, 1 - BC)).
//
// Reordering the topics to line up is read as the one-to-one matching of topics with the
// least total distance.  That linear assignment problem is solved on the host
// (shortest augmenting paths with row and column potentials, the Hungarian
// method of Kuhn and Munkres in O(kp^2 kq)): each augmentation is a chain of
// dependent minimum searches, too sequential to gain from the GPU at the
// topic counts of a topic model.
#include "spdp_internal.hpp"

#include <cmath>
#include <limits>
#include <mutex>
#include <vector>

namespace spdp {

// Partial sums of the allocation-free entry point (spdp_hellinger_noalloc):
// one array per GPU, held until the process ends.  Host code never passes
// this name to a kernel -- on the host it is only a stand-in for the symbol --
// but the device address that hellinger_scratch() looks up once per device.
static __device__ __align__(256) double scratch[kHellingerScratch];

namespace {

constexpr int kTile = 64;     // output tile: kTile x kTile coefficients
constexpr int kStage = 16;    // outcomes per LDS stage (4 MFMA k-steps)
constexpr int kPad = 2;       // LDS row padding (doubles)
constexpr int kThreads = 256; // 4 waves, each a 32 x 32 quarter of the tile

typedef double d4 __attribute__((ext_vector_type(4)));

// part[s][i][j] = sum over outcomes v of slice s of sqrt(P[v][i]) sqrt(Q[v][j])
__global__ void __launch_bounds__(kThreads) k_bc(const double *__restrict__ P, int32_t kp,
                                                 const double *__restrict__ Q, int32_t kq,
                                                 int64_t V, int64_t slice, int32_t tiles_j,
                                                 double *__restrict__ part)
{
    __shared__ double sP[kStage][kTile + kPad], sQ[kStage][kTile + kPad];
    const int32_t i0 = (int32_t)(blockIdx.x / tiles_j) * kTile;
    const int32_t j0 = (int32_t)(blockIdx.x % tiles_j) * kTile;
    const int64_t v_beg = (int64_t)blockIdx.y * slice;
    const int64_t v_end = v_beg + slice < V ? v_beg + slice : V;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wi = (wave >> 1) * 32, wj = (wave & 1) * 32;
    // A operand: lane holds row (lane & 15) of the block at k-step (lane >> 4);
    // B operand: column (lane & 15) at k-step (lane >> 4)
    const int kr = lane >> 4, kc = lane & 15;
    d4 acc00 = {0.0, 0.0, 0.0, 0.0}, acc01 = acc00, acc10 = acc00, acc11 = acc00;

    for (int64_t v0 = v_beg; v0 < v_end; v0 += kStage) {
        for (int e = tid; e < kStage * kTile; e += kThreads) {
            const int r = e / kTile, c = e % kTile;
            const int64_t v = v0 + r;
            const bool in_v = v < v_end;
            sP[r][c] = (in_v && i0 + c < kp) ? sqrt(P[v * kp + i0 + c]) : 0.0;
            sQ[r][c] = (in_v && j0 + c < kq) ? sqrt(Q[v * kq + j0 + c]) : 0.0;
        }
        __syncthreads();
#pragma unroll
        for (int ks = 0; ks < kStage; ks += 4) {
            const double a0 = sP[ks + kr][wi + kc], a1 = sP[ks + kr][wi + 16 + kc];
            const double b0 = sQ[ks + kr][wj + kc], b1 = sQ[ks + kr][wj + 16 + kc];
            acc00 = __builtin_amdgcn_mfma_f64_16x16x4f64(a0, b0, acc00, 0, 0, 0);
            acc01 = __builtin_amdgcn_mfma_f64_16x16x4f64(a0, b1, acc01, 0, 0, 0);
            acc10 = __builtin_amdgcn_mfma_f64_16x16x4f64(a1, b0, acc10, 0, 0, 0);
            acc11 = __builtin_amdgcn_mfma_f64_16x16x4f64(a1, b1, acc11, 0, 0, 0);
        }
        __syncthreads();
    }

    // result block (fp64 layout): value r of a lane is row 4 r + (lane >> 4),
    // column lane & 15
    double *out = part + (int64_t)blockIdx.y * kp * kq;
    const d4 acc[2][2] = {{acc00, acc01}, {acc10, acc11}};
#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
        for (int bj = 0; bj < 2; ++bj)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int32_t i = i0 + wi + bi * 16 + 4 * r + kr;
                const int32_t j = j0 + wj + bj * 16 + kc;
                if (i < kp && j < kq) out[(int64_t)i * kq + j] = acc[bi][bj][r];
            }
}

__global__ void k_hell_finish(int64_t n, int32_t slices, const double *__restrict__ part,
                              double *__restrict__ h)
{
    const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (j >= n) return;
    double bc = 0.0;
    for (int32_t s = 0; s < slices; ++s) bc += part[(int64_t)s * n + j];
    const double d = 1.0 - bc;
    h[j] = sqrt(d > 0.0 ? d : 0.0);
}

}  // namespace

int hellinger_scratch(int device, double **out)
{
    static std::mutex mu;
    static double *addr[kMaxDevices] = {};
    static bool looked_up[kMaxDevices] = {};
    *out = nullptr;
    if (device < 0 || device >= kMaxDevices) return (int)hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (!looked_up[device]) {
        int cur = 0;
        hipError_t e = hipGetDevice(&cur);
        if (e == hipSuccess && cur != device) e = hipSetDevice(device);
        void *p = nullptr;
        if (e == hipSuccess) e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (cur != device) (void)hipSetDevice(cur);
        if (e != hipSuccess) return (int)e;
        addr[device] = static_cast<double *>(p);
        looked_up[device] = true;
    }
    *out = addr[device];
    return (int)hipSuccess;
}

HellingerPlan hellinger_plan(int32_t kp, int32_t kq, int64_t V, int64_t max_part)
{
    HellingerPlan p = hellinger_plan(kp, kq, V);
    const int64_t nh = (int64_t)kp * kq;
    if (nh == 0 || V <= 0) return p;
    int64_t most = max_part / nh;  // slices whose partial sums fit
    if (most < 1) most = 1;
    if (p.slices > most) {
        const int64_t stages = (V + kStage - 1) / kStage;
        const int64_t per = (stages + most - 1) / most;
        p.slice = per * kStage;
        p.slices = (int32_t)((V + p.slice - 1) / p.slice);
    }
    return p;
}

HellingerPlan hellinger_plan(int32_t kp, int32_t kq, int64_t V)
{
    HellingerPlan p;
    const int64_t tiles = (int64_t)((kp + kTile - 1) / kTile) * ((kq + kTile - 1) / kTile);
    const int64_t stages = (V + kStage - 1) / kStage;
    if (tiles == 0) return p;                        // kp or kq = 0: nothing to launch
    int64_t want = (2048 + tiles - 1) / tiles;      // >= 2048 blocks where V allows
    const int64_t most = (stages + 15) / 16;         // >= 16 stages per slice
    if (want > most) want = most;
    if (want < 1) want = 1;
    const int64_t per = (stages + want - 1) / want;  // stages per slice
    p.slice = per * kStage;
    p.slices = (int32_t)(V > 0 ? (V + p.slice - 1) / p.slice : 1);
    p.tiles_j = (kq + kTile - 1) / kTile;
    p.tiles = tiles;
    return p;
}

hipError_t launch_hellinger(const HellingerPlan &p, const double *P, int32_t kp, const double *Q,
                            int32_t kq, int64_t V, double *part, double *h, hipStream_t st)
{
    const int64_t n = (int64_t)kp * kq;
    if (n == 0) return hipSuccess;
    if (V > 0) {
        hipLaunchKernelGGL(k_bc, dim3((unsigned)p.tiles, (unsigned)p.slices), dim3(kThreads), 0,
                           st, P, kp, Q, kq, V, p.slice, p.tiles_j, part);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    const int32_t slices = V > 0 ? p.slices : 0;  // no outcomes: BC = 0, H = 1
    hipLaunchKernelGGL(k_hell_finish, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, n,
                       slices, part, h);
    return hipGetLastError();
}

// Least-total-cost matching of every row of c [kp][kq] (kp <= kq) to its own
// column: for each new row, a shortest augmenting path over the reduced costs
// c[i][j] - u[i] - v[j] (Dijkstra over columns), then the potentials are
// shifted so that matched pairs keep reduced cost 0 and all others stay >= 0.
double align_topics_host(const double *c, int32_t kp, int32_t kq, int32_t *match)
{
    const double inf = std::numeric_limits<double>::infinity();
    // index 0 is a virtual column / row; real rows 1..kp, columns 1..kq
    std::vector<double> u((size_t)kp + 1, 0.0), v((size_t)kq + 1, 0.0), dist((size_t)kq + 1);
    std::vector<int32_t> owner((size_t)kq + 1, 0), prev((size_t)kq + 1, 0);
    std::vector<char> done((size_t)kq + 1);
    for (int32_t row = 1; row <= kp; ++row) {
        owner[0] = row;
        int32_t col = 0;
        std::fill(dist.begin(), dist.end(), inf);
        std::fill(done.begin(), done.end(), 0);
        while (owner[col] != 0) {
            done[col] = 1;
            const int32_t i = owner[col];
            double step = inf;
            int32_t next = 0;
            for (int32_t j = 1; j <= kq; ++j) {
                if (done[j]) continue;
                const double red = c[(int64_t)(i - 1) * kq + (j - 1)] - u[i] - v[j];
                if (red < dist[j]) {
                    dist[j] = red;
                    prev[j] = col;
                }
                if (dist[j] < step) {
                    step = dist[j];
                    next = j;
                }
            }
            for (int32_t j = 0; j <= kq; ++j) {
                if (done[j]) {
                    u[owner[j]] += step;
                    v[j] -= step;
                } else {
                    dist[j] -= step;
                }
            }
            col = next;
        }
        // flip the path: every column on it takes the row of its predecessor
        while (col != 0) {
            const int32_t p = prev[col];
            owner[col] = owner[p];
            col = p;
        }
    }
    double total = 0.0;
    for (int32_t j = 1; j <= kq; ++j)
        if (owner[j] != 0) match[owner[j] - 1] = j - 1;
    for (int32_t i = 0; i < kp; ++i) total += c[(int64_t)i * kq + match[i]];
    return total;
}

}  // namespace spdp
