// Measurement-only kernels: the attainable ceilings that the decode and
// prefill kernels are compared with (they compute nothing of the method).
//
// k_cal_stream reads a buffer with the decode GEMV's weight-stream pattern:
// one contiguous 1 KB tile per wave load (16 bytes per lane, nontemporal),
// two batches of five tiles in flight per wave, 256 workgroups of eight
// waves, consecutive waves on consecutive tiles.  Its time at each decode
// matrix's size is what a pure weight stream of that size costs, launch and
// ramp included.
//
// k_cal_mfma issues v_mfma_f32_16x16x32_bf16 as the prefill GEMM does: 16
// independent accumulators (a 4 x 4 fragment block) per wave, operands in
// registers, loaded once from a buffer whose bit patterns the caller picks
// (random data draws more power than zeros, and the clock follows).
#include <hip/hip_runtime.h>

#include "device_common.h"
#include "pipo.h"

namespace pipo {

constexpr int kCalU = 5;

__global__ __launch_bounds__(512) void k_cal_stream(const u32x4 *__restrict__ w, int64_t ntiles, uint32_t *sink) {
    const int lane = threadIdx.x & 63;
    const int64_t wv = (int64_t)blockIdx.x * 8 + (threadIdx.x >> 6);
    const int64_t nw = (int64_t)gridDim.x * 8;
    const int64_t per = (ntiles + nw - 1) / nw;          // tiles per wave (padded, uniform)
    const int64_t nb = (per + kCalU - 1) / kCalU;        // batches per wave
    auto ptr = [&](int64_t q, int u) -> const u32x4 * {
        const int64_t i = q * kCalU + u, t = wv + i * nw;
        return (i < per && t < ntiles) ? w + t * 64 + lane : w + lane;
    };
    uint32_t acc = 0;
    u32x4 ra[kCalU], rb[kCalU];
#pragma unroll
    for (int u = 0; u < kCalU; ++u) ra[u] = __builtin_nontemporal_load(ptr(0, u));
#pragma unroll
    for (int u = 0; u < kCalU; ++u) rb[u] = __builtin_nontemporal_load(ptr(1, u));
    int64_t q = 0;
    for (; q + 2 < nb; q += 2) {
#pragma unroll
        for (int u = 0; u < kCalU; ++u) acc ^= ra[u][0] ^ ra[u][1] ^ ra[u][2] ^ ra[u][3];
#pragma unroll
        for (int u = 0; u < kCalU; ++u) ra[u] = __builtin_nontemporal_load(ptr(q + 2, u));
#pragma unroll
        for (int u = 0; u < kCalU; ++u) acc ^= rb[u][0] ^ rb[u][1] ^ rb[u][2] ^ rb[u][3];
#pragma unroll
        for (int u = 0; u < kCalU; ++u) rb[u] = __builtin_nontemporal_load(ptr(q + 3, u));
    }
#pragma unroll
    for (int u = 0; u < kCalU; ++u) acc ^= ra[u][0] ^ ra[u][1] ^ ra[u][2] ^ ra[u][3] ^ rb[u][0] ^ rb[u][1] ^ rb[u][2] ^ rb[u][3];
    // the sum is kept alive by a store no real buffer triggers
    if (acc == 0x9e3779b9u) sink[0] = acc;
}

__global__ __launch_bounds__(256) void k_cal_mfma(const u32x4 *__restrict__ ops, int iters, float *sink) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    // eight operand registers per lane, from a 8 KB window of the buffer
    u32x4 a[4], b[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        a[i] = ops[(i * 2) * 64 + lane];
        b[i] = ops[(i * 2 + 1) * 64 + lane];
    }
    f32x4 acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) acc[i][j] = mfma16(a[i], b[j], acc[i][j]);
    }
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) s += acc[i][j][0] + acc[i][j][1] + acc[i][j][2] + acc[i][j][3];
    if (s == 1.2345e-30f) sink[(int)blockIdx.x * 4 + wave] = s;
}

static int n_compute_units() {
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
    return n;
}

// Mean microseconds per launch of launch(r) over `reps` back-to-back launches
// r = 1..reps on stream s (after one untimed launch r = 0).
template <class F>
static int time_launches(F launch, int reps, hipStream_t s, double *us) {
    hipEvent_t e0, e1;
    if (hipEventCreate(&e0) != hipSuccess) return PIPO_EHIP;
    if (hipEventCreate(&e1) != hipSuccess) {
        hipEventDestroy(e0);
        return PIPO_EHIP;
    }
    launch(0);
    hipEventRecord(e0, s);
    for (int r = 1; r <= reps; ++r) launch(r);
    hipEventRecord(e1, s);
    hipError_t e = hipEventSynchronize(e1);
    float ms = 0.f;
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, e0, e1);
    if (e == hipSuccess) e = hipGetLastError();
    hipEventDestroy(e0);
    hipEventDestroy(e1);
    if (e != hipSuccess) return PIPO_EHIP;
    *us = 1000.0 * ms / reps;
    return PIPO_OK;
}

}  // namespace pipo

using namespace pipo;

extern "C" int pipo_calibrate_stream(const void *d_buf, int64_t buf_bytes, int64_t bytes, int32_t reps, double *us,
                                     void *stream) {
    if (!d_buf || !us || bytes < 1024 || bytes % 1024 || buf_bytes < bytes || reps < 1) return PIPO_EINVAL;
    hipStream_t s = (hipStream_t)stream;
    uint32_t *sink = nullptr;
    if (hipMalloc(&sink, 64) != hipSuccess) return PIPO_ENOMEM;
    const int64_t ntiles = bytes / 1024;
    const int64_t span = (buf_bytes - bytes) / 1024 + 1;      // window starts, in 1 KB tiles
    const int rc = time_launches(
        [&](int r) {
            // launch r reads the window at tile (r * ntiles) mod span: consecutive
            // launches read different bytes, so none is served from the caches
            const int64_t t0 = ((int64_t)r * ntiles) % span;
            hipLaunchKernelGGL(k_cal_stream, dim3(256), dim3(512), 0, s, (const u32x4 *)d_buf + t0 * 64, ntiles, sink);
        },
        reps, s, us);
    hipFree(sink);
    return rc;
}

extern "C" int pipo_calibrate_mfma(const void *d_operands, int32_t waves_per_simd, int32_t iters, int32_t reps,
                                   double *tflops, void *stream) {
    if (!d_operands || !tflops || (waves_per_simd != 1 && waves_per_simd != 2 && waves_per_simd != 4) || iters < 1 ||
        reps < 1)
        return PIPO_EINVAL;
    const int ncu = n_compute_units();
    if (ncu <= 0) return PIPO_EHIP;
    hipStream_t s = (hipStream_t)stream;
    const int grid = ncu * waves_per_simd;      // four-wave workgroups: one wave per SIMD each
    float *sink = nullptr;
    if (hipMalloc(&sink, (size_t)grid * 4 * sizeof(float)) != hipSuccess) return PIPO_ENOMEM;
    double us = 0.0;
    const int rc = time_launches(
        [&](int) { hipLaunchKernelGGL(k_cal_mfma, dim3(grid), dim3(256), 0, s, (const u32x4 *)d_operands, iters, sink); },
        reps, s, &us);
    hipFree(sink);
    if (rc != PIPO_OK) return rc;
    const double flops = (double)grid * 4 * iters * 16 * 16384.0;
    *tflops = flops / (us * 1e-6) / 1e12;
    return PIPO_OK;
}
