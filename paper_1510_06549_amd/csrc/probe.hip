// probe.hip -- a read-bandwidth probe of the device (gfx950, wave64): the
// ceiling against which the sampler's bytes per second are read.  Not part of
// the sampling path.
//
//   k_read_seq   the whole buffer once, front to back: grid-stride 16-byte
//                loads, several in flight per lane
//   k_read_rows  one row of row_bytes at a time per wavefront, at
//                pseudo-random row positions (as the sampler reads a token's
//                count row), two rows in flight per wavefront
// Every loaded word enters a per-lane xor, and a lane whose xor equals a value
// that no input here produces stores it, so that no load can be dropped.
#include "spdp_internal.hpp"

namespace spdp {

// the probe's sink: externally visible, so that its stores, and the loads
// they depend on, cannot be dropped
__device__ uint32_t g_probe_sink;

namespace {

constexpr uint32_t kNever = 0x9E3779B9u;

__device__ __forceinline__ uint32_t fold(uint4 v) { return v.x ^ v.y ^ v.z ^ v.w; }

__device__ __forceinline__ void keep(uint32_t acc)
{
    if (acc == kNever) g_probe_sink = acc;
}

__global__ void __launch_bounds__(256) k_read_seq(const uint4 *__restrict__ p, int64_t n)
{
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    uint32_t acc = 0;
    for (; i + 3 * stride < n; i += 4 * stride) {
        const uint4 a = p[i], b = p[i + stride], c = p[i + 2 * stride], d = p[i + 3 * stride];
        acc ^= fold(a) ^ fold(b) ^ fold(c) ^ fold(d);
    }
    for (; i < n; i += stride) acc ^= fold(p[i]);
    keep(acc);
}

// row r of wave w at step i: a 64-bit mix of (w, i), reduced to [0, nrows)
__device__ __forceinline__ int64_t probe_row(uint64_t w, uint64_t i, int64_t nrows)
{
    uint64_t x = (w << 32) ^ i;
    x ^= x >> 33;
    x *= 0xff51afd7ed558ccdull;
    x ^= x >> 33;
    x *= 0xc4ceb9fe1a85ec53ull;
    x ^= x >> 33;
    return (int64_t)(x % (uint64_t)nrows);
}

// CH 16-byte chunks per lane per row (row_bytes = 1024 CH)
template <int CH>
__global__ void __launch_bounds__(64) k_read_rows(const uint4 *__restrict__ p, int64_t nrows,
                                                  int64_t rows_per_wave)
{
    const uint64_t w = blockIdx.x;
    const int32_t lane = threadIdx.x;
    uint32_t acc = 0;
    int64_t i = 0;
    for (; i + 1 < rows_per_wave; i += 2) {
        const uint4 *r0 = p + probe_row(w, i, nrows) * (64 * CH);
        const uint4 *r1 = p + probe_row(w, i + 1, nrows) * (64 * CH);
        uint4 a[CH], b[CH];
#pragma unroll
        for (int c = 0; c < CH; ++c) a[c] = r0[c * 64 + lane];
#pragma unroll
        for (int c = 0; c < CH; ++c) b[c] = r1[c * 64 + lane];
#pragma unroll
        for (int c = 0; c < CH; ++c) acc ^= fold(a[c]) ^ fold(b[c]);
    }
    for (; i < rows_per_wave; ++i) {
        const uint4 *r0 = p + probe_row(w, i, nrows) * (64 * CH);
#pragma unroll
        for (int c = 0; c < CH; ++c) acc ^= fold(r0[c * 64 + lane]);
    }
    keep(acc);
}

template <int CH>
hipError_t launch_rows(const uint4 *p, int64_t nrows, int64_t per_wave, int32_t waves,
                       hipStream_t st)
{
    hipLaunchKernelGGL((k_read_rows<CH>), dim3((unsigned)waves), dim3(64), 0, st, p, nrows,
                       per_wave);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_read_probe(const void *buf, int64_t bytes, int32_t row_bytes, int64_t rows,
                             int32_t waves, hipStream_t st)
{
    const uint4 *p = static_cast<const uint4 *>(buf);
    if (row_bytes == 0) {
        const unsigned blocks = (unsigned)(waves / 4 > 0 ? waves / 4 : 1);
        hipLaunchKernelGGL(k_read_seq, dim3(blocks), dim3(256), 0, st, p, bytes / 16);
        return hipGetLastError();
    }
    const int64_t nrows = bytes / row_bytes;
    const int64_t per_wave = (rows + waves - 1) / waves;
    switch (row_bytes / 1024) {
    case 1: return launch_rows<1>(p, nrows, per_wave, waves, st);
    case 2: return launch_rows<2>(p, nrows, per_wave, waves, st);
    case 3: return launch_rows<3>(p, nrows, per_wave, waves, st);
    case 4: return launch_rows<4>(p, nrows, per_wave, waves, st);
    case 8: return launch_rows<8>(p, nrows, per_wave, waves, st);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace spdp
