// Device-side weight generation and layout packing.
//
// Every weight element is a pure function of (seed, tensor id, logical
// element index): key = sm(seed ^ sm(tid)); r1 = sm(key + 2i), r2 = sm(key +
// 2i + 1); S = sum of the four 24-bit fields r>>40 and (r>>16)&0xFFFFFF;
// w = float(int(S - 2^25)) * 0x1.1bc77ap-29 (both roundings to nearest even),
// an Irwin-Hall(4) variate with sd 0.02; stored as bf16 (nearest even).
//
// Packed row orders (so a 16-row strip holds what one fused epilogue needs):
//   PERM_QK:     inside each head of d rows, strip t holds rows 8t..8t+7 and
//                d/2+8t..d/2+8t+7, the RoPE partners, in its two halves.
//   PERM_GATEUP: strip t holds gate rows 8t..8t+7, then up rows 8t..8t+7.
#include <math.h>
#include "device_common.h"
#include "kernels.h"

namespace pipo {

__device__ __forceinline__ float rspec_value(uint64_t key, uint64_t i) {
    const uint64_t r1 = splitmix64(key + 2ull * i), r2 = splitmix64(key + 2ull * i + 1ull);
    const uint64_t s = (r1 >> 40) + ((r1 >> 16) & 0xFFFFFFull) + (r2 >> 40) + ((r2 >> 16) & 0xFFFFFFull);
    const int32_t c = (int32_t)((int64_t)s - (1ll << 25));
    return __fmul_rn(__int2float_rn(c), __uint_as_float(0x310DE3BDu));
}

// packed local row -> (which tensor, logical row)
__device__ __forceinline__ void unpack_row(int64_t r, int perm, int half, int *which, int64_t *lrow) {
    *which = 0;
    if (perm == PERM_QK) {
        const int64_t d = 2 * half, h = r / d, rr = r - h * d, t = rr >> 4, i = rr & 15;
        *lrow = h * d + (i < 8 ? 8 * t + i : half + 8 * t + (i - 8));
    } else if (perm == PERM_GATEUP) {
        const int64_t t = r >> 4, i = r & 15;
        *which = i < 8 ? 0 : 1;
        *lrow = 8 * t + (i & 7);
    } else {
        *lrow = r;
    }
}

__global__ void k_init_tiled(uint16_t *dst, int64_t K, int64_t row_lo, int64_t nrows, uint64_t seed,
                             uint64_t tid, int perm, int half, uint64_t tid2) {
    const int64_t cpr = K >> 3;
    const int64_t total = nrows * cpr;
    const uint64_t key1 = rng_key(seed, tid), key2 = rng_key(seed, tid2);
    for (int64_t idx = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; idx < total;
         idx += (int64_t)gridDim.x * blockDim.x) {
        const int64_t rl = idx / cpr, k = (idx - rl * cpr) << 3;
        int which;
        int64_t lrow;
        unpack_row(rl, perm, half, &which, &lrow);
        const uint64_t key = which ? key2 : key1;
        const uint64_t base = (uint64_t)(lrow * K + k);
        u32x4 w;
#pragma unroll
        for (int e = 0; e < 4; ++e)
            w[e] = f2bf(rspec_value(key, base + 2 * e)) | (f2bf(rspec_value(key, base + 2 * e + 1)) << 16);
        *(u32x4 *)(dst + tiled_index(row_lo + rl, k, K)) = w;
    }
}

static int grid_for(int64_t total) {
    int64_t g = (total + 255) / 256;
    return (int)(g > 65536 ? 65536 : (g < 1 ? 1 : g));
}

void launch_init_tiled(uint16_t *dst, int64_t N, int64_t K, int64_t row_lo, int64_t row_hi, uint64_t seed,
                       uint64_t tid, int perm, int half, int64_t /*tid_row0*/, uint64_t tid2, hipStream_t s) {
    (void)N;
    const int64_t nrows = row_hi - row_lo;
    hipLaunchKernelGGL(k_init_tiled, dim3(grid_for(nrows * (K >> 3))), dim3(256), 0, s, dst, K, row_lo, nrows,
                       seed, tid, perm, half, tid2);
}

// kind 0: R-spec vector rounded to bf16; 1: gain 1; 2: gain bf16(1 + 10 w)
__global__ void k_init_vec(float *dst, int64_t n, uint64_t seed, uint64_t tid, int kind) {
    const uint64_t key = rng_key(seed, tid);
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
        float v;
        if (kind == 1) v = 1.0f;
        else {
            const float w = rspec_value(key, (uint64_t)i);
            v = kind == 0 ? w : __fadd_rn(1.0f, __fmul_rn(10.0f, w));
            v = bf2f(f2bf(v));
        }
        dst[i] = v;
    }
}

void launch_init_vec(float *dst, int64_t n, uint64_t seed, uint64_t tid, int kind, hipStream_t s) {
    hipLaunchKernelGGL(k_init_vec, dim3(grid_for(n)), dim3(256), 0, s, dst, n, seed, tid, kind);
}

// cos/sin of p * base^(-2j/d), evaluated in double and rounded to float
__global__ void k_rope_table(float *cos_t, float *sin_t, int lmax, int d, double base) {
    const int half = d >> 1;
    const int64_t total = (int64_t)lmax * half;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t pos = i / half;
        const int jj = (int)(i - pos * half);
        const double ang = (double)pos * pow(base, -2.0 * (double)jj / (double)d);
        cos_t[i] = (float)cos(ang);
        sin_t[i] = (float)sin(ang);
    }
}

void launch_rope_table(float *cos_t, float *sin_t, int lmax, int d, double base, hipStream_t s) {
    hipLaunchKernelGGL(k_rope_table, dim3(grid_for((int64_t)lmax * (d >> 1))), dim3(256), 0, s, cos_t, sin_t,
                       lmax, d, base);
}

// logical element -> packed position (inverse of unpack_row), for read-back
__global__ void k_read_tiled(const uint16_t *src, int64_t K, int64_t start, int64_t count, int perm, int half,
                             int64_t row_base, int64_t rows_total, uint16_t *dst) {
    for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < count; t += (int64_t)gridDim.x * blockDim.x) {
        const int64_t e = start + t;
        const int64_t lrow = e / K, k = e - lrow * K;
        int64_t prow;
        if (perm == PERM_QK) {
            const int64_t d = 2 * half, h = lrow / d, rr = lrow - h * d;
            prow = rr < half ? h * d + 16 * (rr >> 3) + (rr & 7) : h * d + 16 * ((rr - half) >> 3) + 8 + ((rr - half) & 7);
        } else if (perm == PERM_GATEUP) {
            // rows [0, rows_total) are gate, [rows_total, 2 rows_total) up
            const int64_t up = lrow >= rows_total ? 1 : 0, r = lrow - up * rows_total;
            prow = 16 * (r >> 3) + 8 * up + (r & 7);
        } else {
            prow = lrow;
        }
        dst[t] = src[tiled_index(row_base + prow, k, K)];
    }
}

void launch_read_tiled(const uint16_t *src, int64_t N, int64_t K, int64_t start, int64_t count, int perm, int half,
                       int64_t row_base, int64_t rows_total, uint16_t *dst, hipStream_t s) {
    (void)N;
    hipLaunchKernelGGL(k_read_tiled, dim3(grid_for(count)), dim3(256), 0, s, src, K, start, count, perm, half,
                       row_base, rows_total, dst);
}

__global__ void k_fill_u32(uint32_t *p, uint32_t v, int64_t n) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) p[i] = v;
}

void launch_fill_u32(uint32_t *p, uint32_t v, int64_t n, hipStream_t s) {
    hipLaunchKernelGGL(k_fill_u32, dim3(grid_for(n)), dim3(256), 0, s, p, v, n);
}

__global__ void k_copy_bytes(uint8_t *dst, const uint8_t *src, int64_t n) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) dst[i] = src[i];
}

void launch_copy_bytes(void *dst, const void *src, int64_t n, hipStream_t s) {
    hipLaunchKernelGGL(k_copy_bytes, dim3(grid_for(n)), dim3(256), 0, s, (uint8_t *)dst, (const uint8_t *)src, n);
}

}  // namespace pipo
