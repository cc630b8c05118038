// Weight-streaming skinny GEMM of the decode step (batch 1..32).
//
// Y^T[N][B] = W[N][K] X^T with W in 16x32 bf16 tiles.  A workgroup of eight
// waves owns SG 16-row strips of W; the waves split the strips' K range
// (wave w takes k-tiles w, w+8, w+16, ...) and stream each tile with one
// contiguous 1 KB load as the MFMA A operand, two batches of loads in flight.
// The activations X (B <= 32 rows) are staged in LDS as the B operand by a
// fused prologue (RMSNorm gain, pair gather, MTP concat), as a pair of bf16
// planes hi + lo (about 16 significant bits; two MFMAs per weight tile, the
// matrix cores have the headroom); the RMSNorm scale is a per-row scalar, so
// it is applied to the accumulators in the epilogue and staging never waits
// for it.  The eight partial sums are reduced through
// LDS in wave order (deterministic, no atomics, no cross-workgroup traffic)
// and a fused epilogue writes the result (bias, residual add, SwiGLU, RoPE +
// KV append, logits + argmax).
#include "device_common.h"
#include "kernels.h"

namespace pipo {

constexpr int kNW = 8;                       // waves per workgroup
constexpr int kGemvLdsBytes = 56 * 1024;     // dynamic LDS budget for the X chunk

__device__ __forceinline__ float silu_f(float u) { return u / (1.0f + __expf(-u)); }

// slot of key kappa (0..31) inside a 32-key V tile; matches the order in which
// the attention kernels hold probabilities as MFMA B operands.
__device__ __forceinline__ int vslot(int kappa) {
    return 8 * ((kappa & 15) >> 2) + 4 * (kappa >> 4) + (kappa & 3);
}

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int m) {
    uint32_t lo = __shfl_xor((uint32_t)v, m), hi = __shfl_xor((uint32_t)(v >> 32), m);
    return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ u32x4 pack8(float4 a, float4 b) {
    u32x4 v;
    v[0] = pack_bf2(a.x, a.y);
    v[1] = pack_bf2(a.z, a.w);
    v[2] = pack_bf2(b.x, b.y);
    v[3] = pack_bf2(b.z, b.w);
    return v;
}

// MTP splits its K range: tiles below H/32 act on RMSNorm(h_b), the rest on
// RMSNorm(E[b]); the two halves get different scales, so they accumulate apart.
template <int PRO>
struct NAcc { static constexpr int n = (PRO == PRO_MTP) ? 2 : 1; };

template <int NBT, int SG, int PRO, int EPI>
__global__ __launch_bounds__(512) void k_gemv(GemvParams p) {
    constexpr int U = 8 / SG;              // k-tiles per wave per load batch
    constexpr int NA = NAcc<PRO>::n;
    constexpr bool HASLO = PRO != PRO_PAIR;   // gathered embeddings are exact in bf16
    extern __shared__ __align__(16) uint16_t xs[];
    __shared__ float sc0[32], sc1[32];

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int j = lane & 15, g = lane >> 4;
    const int nstrips = p.N >> 4;
    const int strip0 = blockIdx.x * SG;
    const int KT = p.K >> 5, HT = p.H >> 5;
    const int B = p.B;
    const int ktpc = p.ktiles_per_chunk;
    const int rstride = ktpc * 32 + 8;
    uint16_t *xs_lo = xs + B * rstride;      // lo plane follows the hi plane

    bool sok[SG];
    const uint16_t *wp[SG];
#pragma unroll
    for (int s = 0; s < SG; ++s) {
        sok[s] = strip0 + s < nstrips;
        wp[s] = p.W + (int64_t)(sok[s] ? strip0 + s : 0) * KT * 512 + lane * 8;
    }

    f32x4 acc[NA][SG][NBT];
#pragma unroll
    for (int a = 0; a < NA; ++a)
#pragma unroll
        for (int s = 0; s < SG; ++s)
#pragma unroll
            for (int bt = 0; bt < NBT; ++bt) acc[a][s][bt] = f32x4{0.f, 0.f, 0.f, 0.f};

    u32x4 ra[2][U][SG];
#pragma unroll
    for (int bsel = 0; bsel < 2; ++bsel)
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int s = 0; s < SG; ++s) ra[bsel][u][s] = u32x4{0u, 0u, 0u, 0u};
    // load batch: k-tiles kt_first + u*8 (u < U) of every strip into ra[BS]
#define GEMV_ISSUE(BS, kt_first, c1)                                                              \
    do {                                                                                          \
        _Pragma("unroll") for (int u = 0; u < U; ++u) {                                           \
            const int kt_ = (kt_first) + u * kNW;                                                 \
            _Pragma("unroll") for (int s = 0; s < SG; ++s) if (kt_ < (c1) && sok[s])              \
                ra[BS][u][s] = __builtin_nontemporal_load((const u32x4 *)(wp[s] + (int64_t)kt_ * 512)); \
        }                                                                                         \
    } while (0)
    // MFMAs of one batch held in ra[BS] against the staged X chunk
#define GEMV_CONSUME(BS, kt_first, c0, c1)                                                        \
    do {                                                                                          \
        _Pragma("unroll") for (int u = 0; u < U; ++u) {                                           \
            const int k2 = (kt_first) + u * kNW;                                                  \
            if (k2 < (c1)) {                                                                      \
                const bool hi_half = NA == 2 && k2 >= HT;                                         \
                _Pragma("unroll") for (int bt = 0; bt < NBT; ++bt) {                              \
                    const int b = bt * 16 + j;                                                    \
                    u32x4 bop = u32x4{0u, 0u, 0u, 0u}, bol = u32x4{0u, 0u, 0u, 0u};               \
                    const int xo = b * rstride + (k2 - (c0)) * 32 + g * 8;                        \
                    if (b < B) {                                                                  \
                        bop = *(const u32x4 *)(xs + xo);                                          \
                        if (HASLO) bol = *(const u32x4 *)(xs_lo + xo);                            \
                    }                                                                             \
                    _Pragma("unroll") for (int s = 0; s < SG; ++s) {                              \
                        f32x4 &ac = hi_half ? acc[NA - 1][s][bt] : acc[0][s][bt];                 \
                        ac = mfma16(ra[BS][u][s], bop, ac);                                       \
                        if (HASLO) ac = mfma16(ra[BS][u][s], bol, ac);                            \
                    }                                                                             \
                }                                                                                 \
            }                                                                                     \
        }                                                                                         \
    } while (0)

    bool scalars_done = false;
    for (int c0 = 0; c0 < KT; c0 += ktpc) {
        const int c1 = min(KT, c0 + ktpc);
        GEMV_ISSUE(0, c0 + wave, c1);          // weights first: independent of the activations
        if (!scalars_done) {
            scalars_done = true;
            if (PRO == PRO_NORM || PRO == PRO_MTP) {
                for (int b = wave; b < B; b += kNW) {
                    float a = 0.f;
                    for (int i = lane; i < p.nss; i += 64) a += p.ss[b * p.nss + i];
                    a = wave_sum(a);
                    const int kn = (PRO == PRO_MTP) ? p.H : p.K;
                    if (lane == 0) sc0[b] = rsqrtf(a / (float)kn + p.eps);
                    if (PRO == PRO_MTP) {
                        const int tok = clamp_id(argmax_key_id(p.tokkey[b]), p.vocab);
                        float e2 = 0.f;
                        for (int k = lane * 8; k < p.H; k += 512) {
                            const u32x4 w = *(const u32x4 *)(p.embed + tiled_index(tok, k, p.H));
#pragma unroll
                            for (int i = 0; i < 4; ++i) {
                                const float lo = bf_lo(w[i]), hi = bf_hi(w[i]);
                                e2 += lo * lo + hi * hi;
                            }
                        }
                        e2 = wave_sum(e2);
                        if (lane == 0) sc1[b] = rsqrtf(e2 / (float)p.H + p.eps);
                    }
                }
            }
        }
        __syncthreads();
        const int cpr = (c1 - c0) * 4;        // 8-element chunks per LDS row
        for (int idx = threadIdx.x; idx < B * cpr; idx += 512) {
            const int b = idx / cpr;
            const int kk = (idx - b * cpr) << 3;
            const int k = c0 * 32 + kk;
            u32x4 vh, vl = u32x4{0u, 0u, 0u, 0u};
            float f[8];
            if (PRO == PRO_PAIR) {
                const bool first = k < p.H;
                const int row = clamp_id(p.pairs[2 * b + (first ? 0 : 1)], p.vocab);
                vh = *(const u32x4 *)(p.embed + tiled_index(row, first ? k : k - p.H, p.H));
            } else {
                if (PRO == PRO_NORM || (PRO == PRO_MTP && k < p.H)) {
                    const int stride = PRO == PRO_MTP ? p.H : p.K;
                    const float4 *xp = (const float4 *)(p.x + (int64_t)b * stride + k);
                    const float4 *gp = (const float4 *)(p.gain + k);
                    const float4 x0 = xp[0], x1 = xp[1], g0 = gp[0], g1 = gp[1];
                    f[0] = x0.x * g0.x; f[1] = x0.y * g0.y; f[2] = x0.z * g0.z; f[3] = x0.w * g0.w;
                    f[4] = x1.x * g1.x; f[5] = x1.y * g1.y; f[6] = x1.z * g1.z; f[7] = x1.w * g1.w;
                } else if (PRO == PRO_F32) {
                    const float4 *xp = (const float4 *)(p.xf + (int64_t)b * p.K + k);
                    const float4 x0 = xp[0], x1 = xp[1];
                    f[0] = x0.x; f[1] = x0.y; f[2] = x0.z; f[3] = x0.w;
                    f[4] = x1.x; f[5] = x1.y; f[6] = x1.z; f[7] = x1.w;
                } else {  // PRO_MTP, second half: E[tok] * g_me
                    const int kh = k - p.H;
                    const int tok = clamp_id(argmax_key_id(p.tokkey[b]), p.vocab);
                    const u32x4 w = *(const u32x4 *)(p.embed + tiled_index(tok, kh, p.H));
                    const float4 *gp = (const float4 *)(p.gain2 + kh);
                    const float4 g0 = gp[0], g1 = gp[1];
                    f[0] = bf_lo(w[0]) * g0.x; f[1] = bf_hi(w[0]) * g0.y; f[2] = bf_lo(w[1]) * g0.z;
                    f[3] = bf_hi(w[1]) * g0.w; f[4] = bf_lo(w[2]) * g1.x; f[5] = bf_hi(w[2]) * g1.y;
                    f[6] = bf_lo(w[3]) * g1.z; f[7] = bf_hi(w[3]) * g1.w;
                }
                split8(f, vh, vl);
            }
            *(u32x4 *)(xs + b * rstride + kk) = vh;
            if (HASLO) *(u32x4 *)(xs_lo + b * rstride + kk) = vl;
        }
        __syncthreads();
        // ping-pong: while one batch is consumed the next is in flight
        int kt = c0 + wave;
        while (kt < c1) {
            int nxt = kt + U * kNW;
            if (nxt < c1) GEMV_ISSUE(1, nxt, c1);
            GEMV_CONSUME(0, kt, c0, c1);
            kt = nxt;
            if (kt >= c1) break;
            nxt = kt + U * kNW;
            if (nxt < c1) GEMV_ISSUE(0, nxt, c1);
            GEMV_CONSUME(1, kt, c0, c1);
            kt = nxt;
        }
    }
#undef GEMV_ISSUE
#undef GEMV_CONSUME

    // ---- reduce the eight waves' partial sums, strip by strip ---------------
    // afterwards wave s < SG holds strip strip0 + s in fin[]
    f32x4 fin[NBT];
#pragma unroll
    for (int bt = 0; bt < NBT; ++bt) fin[bt] = f32x4{0.f, 0.f, 0.f, 0.f};
    f32x4 *red = (f32x4 *)xs;   // [kNW][NBT][64] f32x4, reusing the X chunk
#pragma unroll
    for (int s = 0; s < SG; ++s) {
        __syncthreads();
#pragma unroll
        for (int bt = 0; bt < NBT; ++bt) {
            f32x4 v = acc[0][s][bt];
            if (NA == 2) {
                const int b = bt * 16 + j;
                const float s0 = b < B ? sc0[b] : 0.f, s1 = b < B ? sc1[b] : 0.f;
                v = v * s0 + acc[NA - 1][s][bt] * s1;
            }
            red[(wave * NBT + bt) * 64 + lane] = v;
        }
        __syncthreads();
        if (wave == s) {
#pragma unroll
            for (int bt = 0; bt < NBT; ++bt) {
                f32x4 t = red[bt * 64 + lane];
#pragma unroll
                for (int w = 1; w < kNW; ++w) t += red[(w * NBT + bt) * 64 + lane];
                fin[bt] = t;
            }
        }
    }
    if (wave >= SG) return;
    const int strip = strip0 + wave;
    if (strip >= nstrips) return;
    if (PRO == PRO_NORM) {
#pragma unroll
        for (int bt = 0; bt < NBT; ++bt) {
            const int b = bt * 16 + j;
            fin[bt] *= (b < B ? sc0[b] : 0.f);
        }
    }

    // ---- fused epilogues (one wave per strip) -------------------------------
    const int row0 = strip * 16 + 4 * g;   // first of this lane's four rows
    if (EPI == EPI_STORE || EPI == EPI_RESID) {
#pragma unroll
        for (int bt = 0; bt < NBT; ++bt) {
            const int b = bt * 16 + j;
            const bool ok = b < B;
            f32x4 val = fin[bt];
            float *o = p.out + (int64_t)b * p.N + row0;
            if (ok) {
                if (EPI == EPI_RESID) val += *(const f32x4 *)o;
                else if (p.bias) val += *(const f32x4 *)(p.bias + row0);
                *(f32x4 *)o = val;
            }
            float sq = val[0] * val[0] + val[1] * val[1] + val[2] * val[2] + val[3] * val[3];
            sq = col_sum(sq);
            if (ok && g == 0 && p.ss_out) p.ss_out[b * nstrips + strip] = sq;
        }
    } else if (EPI == EPI_SWIGLU) {
#pragma unroll
        for (int bt = 0; bt < NBT; ++bt) {
            const int b = bt * 16 + j;
            f32x4 up;
#pragma unroll
            for (int v = 0; v < 4; ++v) up[v] = __shfl_xor(fin[bt][v], 32);
            if (b < B && g < 2) {
                const f32x4 ga = fin[bt];
                f32x4 w;
#pragma unroll
                for (int v = 0; v < 4; ++v) w[v] = silu_f(ga[v]) * up[v];
                *(f32x4 *)(p.act + (int64_t)b * (p.N >> 1) + strip * 8 + 4 * g) = w;
            }
        }
    } else if (EPI == EPI_QKV) {
        const int d = p.d, hs = d >> 4;             // strips per head
        const int qs = p.n_q * hs, ks = p.n_kv * hs;
#pragma unroll
        for (int bt = 0; bt < NBT; ++bt) {
            const int b = bt * 16 + j;
            f32x4 other;
#pragma unroll
            for (int v = 0; v < 4; ++v) other[v] = __shfl_xor(fin[bt][v], 32);
            if (b >= B) continue;
            const int pos = p.pos[b];
            if (strip < qs + ks) {
                const bool isq = strip < qs;
                const int sidx = isq ? strip : strip - qs;
                const int head = sidx / hs, t = sidx - head * hs;
                const int jr = 8 * t + 4 * (g & 1);         // rotation index of v = 0
                const int dim0 = (g < 2) ? jr : (d >> 1) + jr;
                const float4 cs = *(const float4 *)(p.rope_cos + (int64_t)pos * (d >> 1) + jr);
                const float4 sn = *(const float4 *)(p.rope_sin + (int64_t)pos * (d >> 1) + jr);
                const float c4[4] = {cs.x, cs.y, cs.z, cs.w}, s4[4] = {sn.x, sn.y, sn.z, sn.w};
                float r[4];
#pragma unroll
                for (int v = 0; v < 4; ++v)
                    r[v] = (g < 2) ? fin[bt][v] * c4[v] - other[v] * s4[v] : fin[bt][v] * c4[v] + other[v] * s4[v];
                u32x2 w;
                w[0] = pack_bf2(r[0], r[1]);
                w[1] = pack_bf2(r[2], r[3]);
                uint16_t *dst = isq ? p.q + ((int64_t)b * p.n_q + head) * d + dim0
                                    : p.kc + (int64_t)b * p.kv_bstride + ((int64_t)head * p.lmax_pad + pos) * d + dim0;
                *(u32x2 *)dst = w;
            } else {
                const int r0 = (strip - qs - ks) * 16 + 4 * g;
                const int kvh = r0 / d, dim = r0 - kvh * d;
                uint16_t *dst = p.vc + (int64_t)b * p.kv_bstride +
                                ((int64_t)(kvh * (p.lmax_pad >> 5) + (pos >> 5)) * d + dim) * 32 + vslot(pos & 31);
#pragma unroll
                for (int v = 0; v < 4; ++v) dst[v * 32] = (uint16_t)f2bf(fin[bt][v]);
            }
        }
    } else if (EPI == EPI_LOGITS) {
#pragma unroll
        for (int bt = 0; bt < NBT; ++bt) {
            const int b = bt * 16 + j;
            const bool ok = b < B;
            if (ok) *(f32x4 *)(p.out + (int64_t)b * p.N + row0) = fin[bt];
            if (p.best) {
                uint64_t key = 0;
                if (ok) {
#pragma unroll
                    for (int v = 0; v < 4; ++v) {
                        const uint64_t kv = argmax_key(fin[bt][v], (uint32_t)(row0 + v));
                        key = kv > key ? kv : key;
                    }
                }
                uint64_t o = shfl_xor_u64(key, 16);
                key = o > key ? o : key;
                o = shfl_xor_u64(key, 32);
                key = o > key ? o : key;
                if (g == 0 && ok) atomicMax((unsigned long long *)(p.best + b), (unsigned long long)key);
            }
        }
    }
}

template <int NBT, int SG, int PRO, int EPI>
static void launch_t(const GemvParams &p, hipStream_t s) {
    GemvParams q = p;
    const int KT = q.K >> 5;
    constexpr int planes = PRO == PRO_PAIR ? 1 : 2;
    int ktpc = (kGemvLdsBytes / (2 * planes) / q.B - 8) / 32;
    ktpc = ktpc > KT ? KT : ktpc;
    q.ktiles_per_chunk = ktpc;
    int lds = planes * q.B * (ktpc * 32 + 8) * 2;
    const int red = kNW * NBT * 64 * 16;
    lds = lds > red ? lds : red;
    const int grid = ((q.N >> 4) + SG - 1) / SG;
    hipLaunchKernelGGL((k_gemv<NBT, SG, PRO, EPI>), dim3(grid), dim3(kNW * 64), lds, s, q);
}

template <int SG, int PRO, int EPI>
static void launch_nbt(const GemvParams &p, hipStream_t s) {
    if (p.B <= 16) launch_t<1, SG, PRO, EPI>(p, s);
    else launch_t<2, SG, PRO, EPI>(p, s);
}

// One instantiation per (prologue, epilogue) pair the decode step uses; the
// strips per workgroup follow the matrix height: the LM head (151936 rows)
// and gate/up (19456) take 4 and 2 strips, the rest one.
void launch_gemv(const GemvParams &p, int pro, int epi, hipStream_t s) {
    if (pro == PRO_PAIR && epi == EPI_STORE) launch_nbt<1, PRO_PAIR, EPI_STORE>(p, s);
    else if (pro == PRO_NORM && epi == EPI_QKV) launch_nbt<1, PRO_NORM, EPI_QKV>(p, s);
    else if (pro == PRO_F32 && epi == EPI_RESID) launch_nbt<1, PRO_F32, EPI_RESID>(p, s);
    else if (pro == PRO_NORM && epi == EPI_SWIGLU) launch_nbt<2, PRO_NORM, EPI_SWIGLU>(p, s);
    else if (pro == PRO_NORM && epi == EPI_LOGITS) launch_nbt<4, PRO_NORM, EPI_LOGITS>(p, s);
    else if (pro == PRO_MTP && epi == EPI_STORE) launch_nbt<1, PRO_MTP, EPI_STORE>(p, s);
    else if (pro == PRO_NORM && epi == EPI_STORE) launch_nbt<1, PRO_NORM, EPI_STORE>(p, s);
}

}  // namespace pipo
