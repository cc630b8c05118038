// Weight-streaming skinny GEMM of the decode step (batch 1..32).
//
// Y^T[N][B] = W[N][K] X^T with W in 16x32 bf16 tiles: each wave owns one
// 16-row strip of W and streams it tile by tile (one contiguous 1 KB load per
// tile) as the MFMA A operand; the activations X (B <= 32 rows) are produced
// once per workgroup into LDS by a fused prologue (RMSNorm, pair gather, MTP
// concat) and read as the B operand.  Small-N matrices are split along K; the
// last workgroup of a strip group to finish sums the partials in split order
// (deterministic) and runs the fused epilogue (bias, residual add, SwiGLU,
// RoPE + KV append, logits + argmax).
#include "device_common.h"
#include "kernels.h"

namespace pipo {

constexpr int kGemvWaves = 4;
constexpr int kGemvUnroll = 8;
constexpr int kGemvLdsBytes = 48 * 1024;   // dynamic LDS budget; static LDS adds ~1.2 KB

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

template <int NBT, int PRO, int EPI>
__global__ __launch_bounds__(256) void k_gemv(GemvParams p) {
    extern __shared__ __align__(16) uint16_t xs[];
    __shared__ float sc0[32], sc1[32];
    __shared__ int s_last;
    __shared__ uint64_t s_best[kGemvWaves][32];

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int j = lane & 15, g = lane >> 4;
    const int nstrips = p.N >> 4;
    const int groups = (nstrips + kGemvWaves - 1) / kGemvWaves;
    const int grp = blockIdx.x % groups;
    const int split = blockIdx.x / groups;
    const int KT = p.K >> 5;
    const int ktps = (KT + p.splits - 1) / p.splits;
    const int kt0 = split * ktps;
    const int kt1 = min(KT, kt0 + ktps);
    const int strip = grp * kGemvWaves + wave;
    const bool strip_ok = strip < nstrips;
    const int B = p.B;
    const int rstride = p.ktiles_per_chunk * 32 + 8;

    if (PRO == PRO_NORM || PRO == PRO_MTP) {
        for (int b = wave; b < B; b += kGemvWaves) {
            float a = 0.f;
            for (int i = lane; i < p.nss; i += 64) a += p.ss[b * p.nss + i];
            a = wave_sum(a);
            const int kn = (PRO == PRO_MTP) ? p.H : p.K;
            if (lane == 0) sc0[b] = rsqrtf(a / (float)kn + p.eps);
            if (PRO == PRO_MTP) {
                const int tok = clamp_id(argmax_key_id(p.tokkey[b]), p.vocab);
                float e2 = 0.f;
                for (int k = lane * 8; k < p.H; k += 512) {
                    u32x4 w = *(const u32x4 *)(p.embed + tiled_index(tok, k, p.H));
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        float lo = bf_lo(w[i]), hi = bf_hi(w[i]);
                        e2 += lo * lo + hi * hi;
                    }
                }
                e2 = wave_sum(e2);
                if (lane == 0) sc1[b] = rsqrtf(e2 / (float)p.H + p.eps);
            }
        }
    }

    f32x4 acc[NBT];
#pragma unroll
    for (int bt = 0; bt < NBT; ++bt) acc[bt] = f32x4{0.f, 0.f, 0.f, 0.f};

    const uint16_t *wstrip = p.W + (int64_t)strip * KT * 512 + lane * 8;

    for (int c0 = kt0; c0 < kt1; c0 += p.ktiles_per_chunk) {
        const int c1 = min(kt1, c0 + p.ktiles_per_chunk);
        const int cpr = (c1 - c0) * 4;   // 8-element chunks per LDS row
        __syncthreads();
        for (int idx = threadIdx.x; idx < B * cpr; idx += 256) {
            const int b = idx / cpr;
            const int kk = (idx - b * cpr) << 3;
            const int k = c0 * 32 + kk;
            u32x4 v;
            if (PRO == PRO_NORM) {
                const float4 *xp = (const float4 *)(p.x + (int64_t)b * p.K + k);
                const float4 *gp = (const float4 *)(p.gain + k);
                const float4 x0 = xp[0], x1 = xp[1], g0 = gp[0], g1 = gp[1];
                const float s = sc0[b];
                v[0] = pack_bf2(x0.x * s * g0.x, x0.y * s * g0.y);
                v[1] = pack_bf2(x0.z * s * g0.z, x0.w * s * g0.w);
                v[2] = pack_bf2(x1.x * s * g1.x, x1.y * s * g1.y);
                v[3] = pack_bf2(x1.z * s * g1.z, x1.w * s * g1.w);
            } else if (PRO == PRO_BF16) {
                v = *(const u32x4 *)(p.xb + (int64_t)b * p.K + k);
            } else if (PRO == PRO_PAIR) {
                const bool first = k < p.H;
                const int row = clamp_id(p.pairs[2 * b + (first ? 0 : 1)], p.vocab);
                v = *(const u32x4 *)(p.embed + tiled_index(row, first ? k : k - p.H, p.H));
            } else {  // PRO_MTP
                if (k < p.H) {
                    const float4 *xp = (const float4 *)(p.x + (int64_t)b * p.H + k);
                    const float4 *gp = (const float4 *)(p.gain + k);
                    const float4 x0 = xp[0], x1 = xp[1], g0 = gp[0], g1 = gp[1];
                    const float s = sc0[b];
                    v[0] = pack_bf2(x0.x * s * g0.x, x0.y * s * g0.y);
                    v[1] = pack_bf2(x0.z * s * g0.z, x0.w * s * g0.w);
                    v[2] = pack_bf2(x1.x * s * g1.x, x1.y * s * g1.y);
                    v[3] = pack_bf2(x1.z * s * g1.z, x1.w * s * g1.w);
                } else {
                    const int kh = k - p.H;
                    const int tok = clamp_id(argmax_key_id(p.tokkey[b]), p.vocab);
                    const u32x4 w = *(const u32x4 *)(p.embed + tiled_index(tok, kh, p.H));
                    const float4 *gp = (const float4 *)(p.gain2 + kh);
                    const float4 g0 = gp[0], g1 = gp[1];
                    const float s = sc1[b];
                    v[0] = pack_bf2(bf_lo(w[0]) * s * g0.x, bf_hi(w[0]) * s * g0.y);
                    v[1] = pack_bf2(bf_lo(w[1]) * s * g0.z, bf_hi(w[1]) * s * g0.w);
                    v[2] = pack_bf2(bf_lo(w[2]) * s * g1.x, bf_hi(w[2]) * s * g1.y);
                    v[3] = pack_bf2(bf_lo(w[3]) * s * g1.z, bf_hi(w[3]) * s * g1.w);
                }
            }
            *(u32x4 *)(xs + b * rstride + kk) = v;
        }
        __syncthreads();
        if (strip_ok) {
            int kt = c0;
            for (; kt + kGemvUnroll <= c1; kt += kGemvUnroll) {
                u32x4 a[kGemvUnroll];
#pragma unroll
                for (int u = 0; u < kGemvUnroll; ++u)
                    a[u] = __builtin_nontemporal_load((const u32x4 *)(wstrip + (int64_t)(kt + u) * 512));
#pragma unroll
                for (int u = 0; u < kGemvUnroll; ++u) {
#pragma unroll
                    for (int bt = 0; bt < NBT; ++bt) {
                        const int b = bt * 16 + j;
                        u32x4 bop = u32x4{0u, 0u, 0u, 0u};
                        if (b < B) bop = *(const u32x4 *)(xs + b * rstride + (kt + u - c0) * 32 + g * 8);
                        acc[bt] = mfma16(a[u], bop, acc[bt]);
                    }
                }
            }
            for (; kt < c1; ++kt) {
                const u32x4 a = __builtin_nontemporal_load((const u32x4 *)(wstrip + (int64_t)kt * 512));
#pragma unroll
                for (int bt = 0; bt < NBT; ++bt) {
                    const int b = bt * 16 + j;
                    u32x4 bop = u32x4{0u, 0u, 0u, 0u};
                    if (b < B) bop = *(const u32x4 *)(xs + b * rstride + (kt - c0) * 32 + g * 8);
                    acc[bt] = mfma16(a, bop, acc[bt]);
                }
            }
        }
    }

    // ---- split-K: the last arriving workgroup of this strip group reduces --
    if (p.splits > 1) {
        if (strip_ok) {
#pragma unroll
            for (int bt = 0; bt < NBT; ++bt) {
                const int b = bt * 16 + j;
                if (b < B)
                    *(f32x4 *)(p.part + ((int64_t)split * B + b) * p.N + strip * 16 + 4 * g) = acc[bt];
            }
        }
        __threadfence();
        __syncthreads();
        if (threadIdx.x == 0) {
            const uint32_t prev = __hip_atomic_fetch_add(p.ctr + grp, 1u, __ATOMIC_ACQ_REL,
                                                         __HIP_MEMORY_SCOPE_AGENT);
            s_last = (prev == (uint32_t)(p.splits - 1));
        }
        __syncthreads();
        if (!s_last) return;
        __threadfence();
        if (strip_ok) {
#pragma unroll
            for (int bt = 0; bt < NBT; ++bt) {
                const int b = bt * 16 + j;
                f32x4 s = f32x4{0.f, 0.f, 0.f, 0.f};
                if (b < B) {
                    for (int sp = 0; sp < p.splits; ++sp)
                        s += *(const f32x4 *)(p.part + ((int64_t)sp * B + b) * p.N + strip * 16 + 4 * g);
                }
                acc[bt] = s;
            }
        }
        if (threadIdx.x == 0) p.ctr[grp] = 0u;
    }

    // ---- fused epilogues ----------------------------------------------------
    const int row0 = strip * 16 + 4 * g;   // first of this lane's four rows
    if (EPI == EPI_STORE || EPI == EPI_RESID) {
#pragma unroll
        for (int bt = 0; bt < NBT; ++bt) {
            const int b = bt * 16 + j;
            const bool ok = strip_ok && b < B;
            f32x4 val = acc[bt];
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
            for (int v = 0; v < 4; ++v) up[v] = __shfl_xor(acc[bt][v], 32);
            if (strip_ok && b < B && g < 2) {
                const f32x4 ga = acc[bt];
                u32x2 w;
                w[0] = pack_bf2(silu_f(ga[0]) * up[0], silu_f(ga[1]) * up[1]);
                w[1] = pack_bf2(silu_f(ga[2]) * up[2], silu_f(ga[3]) * up[3]);
                *(u32x2 *)(p.act + (int64_t)b * (p.N >> 1) + strip * 8 + 4 * g) = w;
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
            for (int v = 0; v < 4; ++v) other[v] = __shfl_xor(acc[bt][v], 32);
            if (!strip_ok || b >= B) continue;
            const int pos = p.pos[b];
            if (strip < qs + ks) {
                const bool isq = strip < qs;
                const int sidx = isq ? strip : strip - qs;
                const int head = sidx / hs, t = sidx - head * hs;
                const int jr = 8 * t + 4 * (g & 1);         // rotation index of v = 0
                const int dim0 = (g < 2) ? jr : (d >> 1) + jr;
                const float *cs = p.rope_cos + (int64_t)pos * (d >> 1) + jr;
                const float *sn = p.rope_sin + (int64_t)pos * (d >> 1) + jr;
                float r[4];
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const float c = cs[v], s = sn[v];
                    r[v] = (g < 2) ? acc[bt][v] * c - other[v] * s : acc[bt][v] * c + other[v] * s;
                }
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
                for (int v = 0; v < 4; ++v) dst[v * 32] = (uint16_t)f2bf(acc[bt][v]);
            }
        }
    } else if (EPI == EPI_LOGITS) {
#pragma unroll
        for (int bt = 0; bt < NBT; ++bt) {
            const int b = bt * 16 + j;
            const bool ok = strip_ok && b < B;
            if (ok) *(f32x4 *)(p.out + (int64_t)b * p.N + row0) = acc[bt];
            if (p.best) {
                uint64_t key = 0;
                if (ok) {
#pragma unroll
                    for (int v = 0; v < 4; ++v) {
                        const uint64_t kv = argmax_key(acc[bt][v], (uint32_t)(row0 + v));
                        key = kv > key ? kv : key;
                    }
                }
                uint64_t o = shfl_xor_u64(key, 16);
                key = o > key ? o : key;
                o = shfl_xor_u64(key, 32);
                key = o > key ? o : key;
                if (g == 0) s_best[wave][bt * 16 + j] = key;
            }
        }
        if (p.best) {
            __syncthreads();
            if (threadIdx.x < B) {
                uint64_t m = s_best[0][threadIdx.x];
#pragma unroll
                for (int w = 1; w < kGemvWaves; ++w) m = s_best[w][threadIdx.x] > m ? s_best[w][threadIdx.x] : m;
                if (m) atomicMax((unsigned long long *)(p.best + threadIdx.x), (unsigned long long)m);
            }
        }
    }
}

int gemv_num_groups(int N) { return ((N >> 4) + kGemvWaves - 1) / kGemvWaves; }

template <int NBT, int PRO, int EPI>
static void launch_t(const GemvParams &p, int grid, int lds, hipStream_t s) {
    hipLaunchKernelGGL((k_gemv<NBT, PRO, EPI>), dim3(grid), dim3(256), lds, s, p);
}

template <int NBT, int PRO>
static void launch_epi(const GemvParams &p, int epi, int grid, int lds, hipStream_t s) {
    switch (epi) {
        case EPI_STORE: launch_t<NBT, PRO, EPI_STORE>(p, grid, lds, s); break;
        case EPI_RESID: launch_t<NBT, PRO, EPI_RESID>(p, grid, lds, s); break;
        case EPI_SWIGLU: launch_t<NBT, PRO, EPI_SWIGLU>(p, grid, lds, s); break;
        case EPI_QKV: launch_t<NBT, PRO, EPI_QKV>(p, grid, lds, s); break;
        default: launch_t<NBT, PRO, EPI_LOGITS>(p, grid, lds, s); break;
    }
}

template <int NBT>
static void launch_pro(const GemvParams &p, int pro, int epi, int grid, int lds, hipStream_t s) {
    switch (pro) {
        case PRO_NORM: launch_epi<NBT, PRO_NORM>(p, epi, grid, lds, s); break;
        case PRO_BF16: launch_epi<NBT, PRO_BF16>(p, epi, grid, lds, s); break;
        case PRO_PAIR: launch_epi<NBT, PRO_PAIR>(p, epi, grid, lds, s); break;
        default: launch_epi<NBT, PRO_MTP>(p, epi, grid, lds, s); break;
    }
}

// The caller fills everything but splits / ktiles_per_chunk, which depend on
// the shape: enough workgroups to cover the CUs twice, at least 4 k-tiles per
// split, at most 16 splits (the partial buffer's size).
void launch_gemv(const GemvParams &p0, int pro, int epi, hipStream_t s) {
    GemvParams p = p0;
    const int KT = p.K >> 5;
    const int groups = gemv_num_groups(p.N);
    int splits = 1;
    if (epi != EPI_LOGITS) {
        splits = (512 + groups - 1) / groups;
        splits = splits < 1 ? 1 : splits;
        splits = splits > 16 ? 16 : splits;
        while (splits > 1 && KT / splits < 4) --splits;
    }
    p.splits = splits;
    const int ktps = (KT + splits - 1) / splits;
    int ktpc = (kGemvLdsBytes / 2 / p.B - 8) / 32;
    ktpc = ktpc > ktps ? ktps : ktpc;
    p.ktiles_per_chunk = ktpc;
    const int lds = p.B * (ktpc * 32 + 8) * 2;
    const int grid = groups * splits;
    if (p.B <= 16) launch_pro<1>(p, pro, epi, grid, lds, s);
    else launch_pro<2>(p, pro, epi, grid, lds, s);
}

}  // namespace pipo
