// Weight-streaming skinny GEMM of the decode step (batch 1..32).
//
// Y^T[N][B] = W[N][K] X^T with W in 16x32 bf16 tiles.  A strip group is 8/KS
// 16-row strips of W handled by the eight waves of a workgroup, KS waves per
// strip splitting its K range (wave k of a strip takes k-tiles k, k+KS,
// k+2KS, ...); every wave streams its tiles with one contiguous 1 KB load
// each as the MFMA A operand.  KS is chosen per matrix: tall matrices (the LM
// head) give every wave a whole strip, short ones split K to keep enough
// loads in flight.  The layer matrices run one workgroup per compute unit,
// each taking every n-th strip group in one continuous weight stream (this
// evens out the tail of the 1216-strip gate/up matrix).
//
// Memory operations retire in issue order, so a wave first loads what the
// prologue and epilogue need (the activation sources of the first LDS chunk,
// RMSNorm partial sums, the residual rows), then issues two batches of weight
// tiles, and only then waits: staging X in LDS never waits for weights, and
// the weight stream never drains behind the prologue.  X is staged as a pair
// of bf16 planes hi + lo (about 16 significant bits; two MFMAs per weight
// tile, the matrix cores have the headroom).  The RMSNorm scale is a per-row
// scalar applied to the accumulators in the epilogue.  The KS partial sums of
// a strip are reduced through LDS in wave order (deterministic, no atomics,
// no cross-workgroup traffic) and a fused epilogue writes the result (bias,
// residual add, SwiGLU, RoPE + KV append, logits + argmax).
#include <hip/hip_ext.h>

#include <algorithm>

#include "device_common.h"
#include "kernels.h"

namespace pipo {

thread_local GemvTiming g_gemv_timing = {nullptr, nullptr, false};

constexpr int kNW = 8;                       // waves per workgroup
constexpr int kMaxB = 64;                    // columns (sequences) at most: four 16-column tiles
constexpr int kGemvOneLdsBytes = 72 * 1024;  // budget for wave-private X (two workgroups per CU)
// The residual and SwiGLU epilogues may take one workgroup per CU instead
// (X up to 150 KB, e.g. 8 rows of K = 4096): no k-ranges, so no finishing
// launch (9B at batch 8: pair step 6.03 -> 5.96 ms).  QKV keeps the k-range
// path there, whose finish the decode attention takes over.
constexpr int kGemvOneLdsBytesWide = 150 * 1024;
// k-tiles per shared X chunk (larger batches); beyond 32 columns half as
// many, so that the X and weight registers of two chunks in flight fit
constexpr int wide_chunk(int nbt) { return nbt <= 2 ? 8 : 4; }
constexpr int kXR = 3;                       // prologue chunks per thread loaded ahead of the weights

__device__ __forceinline__ float silu_f(float u) { return u / (1.0f + __expf(-u)); }


__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int m) {
    uint32_t lo = __shfl_xor((uint32_t)v, m), hi = __shfl_xor((uint32_t)(v >> 32), m);
    return ((uint64_t)hi << 32) | lo;
}

// The raw inputs of one 8-element prologue chunk, loaded early.
struct XSrc {
    float4 a0, a1;   // x (or x_f)
    float4 g0, g1;   // gain
    u32x4 e;         // gathered bf16 embedding
};

// MTP splits its K range: tiles below H/32 act on RMSNorm(h_b), the rest on
// RMSNorm(E[b]); the two halves get different scales, so they accumulate apart.
template <int PRO>
struct NAcc { static constexpr int n = (PRO == PRO_MTP) ? 2 : 1; };

template <int PRO>
__device__ __forceinline__ void load_src(const GemvParams &p, int b, int k, XSrc &s) {
    if (PRO == PRO_PAIR) {
        const bool first = k < p.H;
        const int row = clamp_id(p.pairs[2 * b + (first ? 0 : 1)], p.vocab);
        s.e = *(const u32x4 *)(p.embed + tiled_index(row, first ? k : k - p.H, p.H));
    } else if (PRO == PRO_F32) {
        const float4 *xp = (const float4 *)(p.xf + (int64_t)b * p.K + k);
        s.a0 = xp[0];
        s.a1 = xp[1];
    } else if (PRO == PRO_CAT) {   // [x; x2] * gain over 2H
        const float4 *xp = (const float4 *)(k < p.H ? p.x + (int64_t)b * p.H + k : p.x2 + (int64_t)b * p.H + k - p.H);
        const float4 *gp = (const float4 *)(p.gain + k);
        s.a0 = xp[0];
        s.a1 = xp[1];
        s.g0 = gp[0];
        s.g1 = gp[1];
    } else if (PRO == PRO_NORM || k < p.H) {
        const int stride = PRO == PRO_MTP ? p.H : p.K;
        const float4 *xp = (const float4 *)(p.x + (int64_t)b * stride + k);
        const float4 *gp = (const float4 *)(p.gain + k);
        s.a0 = xp[0];
        s.a1 = xp[1];
        s.g0 = gp[0];
        s.g1 = gp[1];
    } else {   // PRO_MTP, second half: E[tok] * g_me
        const int kh = k - p.H;
        const int tok = clamp_id(argmax_key_id(p.tokkey[b]), p.vocab);
        s.e = *(const u32x4 *)(p.embed + tiled_index(tok, kh, p.H));
        const float4 *gp = (const float4 *)(p.gain2 + kh);
        s.g0 = gp[0];
        s.g1 = gp[1];
    }
}

// hi / lo bf16 words of one chunk from its raw inputs
template <int PRO>
__device__ __forceinline__ void make_chunk(const GemvParams &p, int k, const XSrc &s, u32x4 &vh, u32x4 &vl) {
    if (PRO == PRO_PAIR) {
        vh = s.e;
        vl = u32x4{0u, 0u, 0u, 0u};
        return;
    }
    float f[8];
    if (PRO == PRO_F32) {
        f[0] = s.a0.x; f[1] = s.a0.y; f[2] = s.a0.z; f[3] = s.a0.w;
        f[4] = s.a1.x; f[5] = s.a1.y; f[6] = s.a1.z; f[7] = s.a1.w;
    } else if (PRO == PRO_NORM || PRO == PRO_CAT || k < p.H) {
        f[0] = s.a0.x * s.g0.x; f[1] = s.a0.y * s.g0.y; f[2] = s.a0.z * s.g0.z; f[3] = s.a0.w * s.g0.w;
        f[4] = s.a1.x * s.g1.x; f[5] = s.a1.y * s.g1.y; f[6] = s.a1.z * s.g1.z; f[7] = s.a1.w * s.g1.w;
    } else {
        f[0] = bf_lo(s.e[0]) * s.g0.x; f[1] = bf_hi(s.e[0]) * s.g0.y; f[2] = bf_lo(s.e[1]) * s.g0.z;
        f[3] = bf_hi(s.e[1]) * s.g0.w; f[4] = bf_lo(s.e[2]) * s.g1.x; f[5] = bf_hi(s.e[2]) * s.g1.y;
        f[6] = bf_lo(s.e[3]) * s.g1.z; f[7] = bf_hi(s.e[3]) * s.g1.w;
    }
    split8(f, vh, vl);
}

// Where the 8-element chunks of X go in LDS.
//  shared (several LDS chunks, large batch): the workgroup stages columns
//    [32 c0, 32 c1) of every row cooperatively, row b at b * rstride.
//  private (X fits): wave (strip, ks) multiplies only k-tiles ks + KS i, so it
//    stages exactly those 32-column slices in its own region, row b at
//    b * rstride, slice i at 32 i; no other wave reads them and no workgroup
//    barrier is needed before the first MFMA.
struct ChunkMap {
    bool priv;
    int per_row;        // chunks per row
    int count;          // chunks in total
    int ks, KS, KT;     // private: this wave's k-split
    int rstride;
    __device__ __forceinline__ int first() const { return priv ? (threadIdx.x & 63) : threadIdx.x; }
    __device__ __forceinline__ int step() const { return priv ? 64 : 512; }
    // chunk idx -> row b, global column k, LDS element offset (relative to the plane base)
    __device__ __forceinline__ void map(int idx, int &b, int &k, int &off) const {
        b = idx / per_row;
        const int rem = idx - b * per_row;
        if (priv) {
            const int i = rem >> 2, q = rem & 3;
            const int kt = ks + KS * i;
            k = (kt < KT ? kt * 32 : 0) + q * 8;
            off = b * rstride + i * 32 + q * 8;
        } else {
            k = rem << 3;
            off = b * rstride + k;
        }
    }
};

// Prologue: everything the first LDS chunk, the RMSNorm scalars and the
// residual epilogue read, issued as unconditional loads (out-of-range indices
// are clamped and the values discarded) so that the compiler's wait counts
// stay exact and never cover the weight loads issued after them.
template <int NBT, int PRO, int EPI>
struct Pro {
    static constexpr int RPW = 2 * NBT;    // RMSNorm rows per wave: b = wave + 8 r
    f32x4 resid[NBT];
    float ssv[RPW][4];                     // sum-of-squares parts, 4 per lane (nss <= 256)
    float ssv2[PRO == PRO_CAT ? RPW : 1][4];   // PRO_CAT: the second half's parts
    XSrc src[kXR];
};

template <int NBT, int PRO, int EPI>
__device__ __forceinline__ void pro_load(const GemvParams &p, Pro<NBT, PRO, EPI> &pr, bool lead,
                                         int row0, const ChunkMap &cm, int col0) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, j = lane & 15;
    constexpr bool NORM = PRO == PRO_NORM || PRO == PRO_MTP || PRO == PRO_CAT;
#pragma unroll
    for (int bt = 0; bt < NBT; ++bt) {
        const int b = bt * 16 + j;
        if (EPI == EPI_RESID)
            pr.resid[bt] = *(const f32x4 *)(p.out + ((lead && b < p.B) ? (int64_t)b * p.N + row0 : 0));
    }
    if (NORM) {
#pragma unroll
        for (int r = 0; r < Pro<NBT, PRO, EPI>::RPW; ++r)
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                const int b = wave + r * kNW, i = lane + 64 * t;
                pr.ssv[r][t] = p.ss[(b < p.B && i < p.nss) ? b * p.nss + i : 0];
                if (PRO == PRO_CAT) pr.ssv2[r][t] = p.ss2[(b < p.B && i < p.nss) ? b * p.nss + i : 0];
            }
    }
#pragma unroll
    for (int r = 0; r < kXR; ++r) {
        int idx = cm.first() + r * cm.step();
        idx = idx < cm.count ? idx : 0;
        int b, k, off;
        cm.map(idx, b, k, off);
        load_src<PRO>(p, b, col0 + k, pr.src[r]);
    }
}

// RMSNorm scalars into sc0 (and sc1 for the MTP's embedding half), then the
// chunks of X this thread loaded (and any beyond kXR per thread).
template <int NBT, int PRO, int EPI>
__device__ __forceinline__ void pro_finish(const GemvParams &p, const Pro<NBT, PRO, EPI> &pr, const ChunkMap &cm,
                                           int col0, uint16_t *xh, uint16_t *xl, float *sc0, float *sc1) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    constexpr bool NORM = PRO == PRO_NORM || PRO == PRO_MTP || PRO == PRO_CAT;
    constexpr bool HASLO = PRO != PRO_PAIR;
    const int B = p.B;
    if (NORM) {
#pragma unroll
        for (int r = 0; r < Pro<NBT, PRO, EPI>::RPW; ++r) {
            const int b = wave + r * kNW;
            float a = 0.f;
#pragma unroll
            for (int t = 0; t < 4; ++t) a += (lane + 64 * t < p.nss) ? pr.ssv[r][t] : 0.f;
            if (PRO == PRO_CAT) {
#pragma unroll
                for (int t = 0; t < 4; ++t) a += (lane + 64 * t < p.nss) ? pr.ssv2[r][t] : 0.f;
            }
            a = wave_sum_dpp(a);
            if (b < B && lane == 0) sc0[b] = rsqrtf(a / (float)(PRO == PRO_MTP ? p.H : p.K) + p.eps);
        }
    }
    if (PRO == PRO_MTP) {
        // RMSNorm scale of E[tok] (a short row, read here after the weights)
        for (int b = wave; b < B; b += kNW) {
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
            e2 = wave_sum_dpp(e2);
            if (lane == 0) sc1[b] = rsqrtf(e2 / (float)p.H + p.eps);
        }
    }
#pragma unroll
    for (int r = 0; r < kXR; ++r) {
        const int idx = cm.first() + r * cm.step();
        if (idx < cm.count) {
            int b, k, off;
            cm.map(idx, b, k, off);
            u32x4 vh, vl;
            make_chunk<PRO>(p, col0 + k, pr.src[r], vh, vl);
            *(u32x4 *)(xh + off) = vh;
            if (HASLO) *(u32x4 *)(xl + off) = vl;
        }
    }
    for (int idx = cm.first() + kXR * cm.step(); idx < cm.count; idx += cm.step()) {   // large B only
        int b, k, off;
        cm.map(idx, b, k, off);
        XSrc sx;
        load_src<PRO>(p, b, col0 + k, sx);
        u32x4 vh, vl;
        make_chunk<PRO>(p, col0 + k, sx, vh, vl);
        *(u32x4 *)(xh + off) = vh;
        if (HASLO) *(u32x4 *)(xl + off) = vl;
    }
}

// acc += W tile x X^T chunk for one 1 KB weight tile: kt is its k-tile, xcol
// the LDS column where its 32 columns of X start; w is already zero for
// padding tiles.
template <int NBT, int PRO>
__device__ __forceinline__ void tile_mma(f32x4 (&acc)[NAcc<PRO>::n][NBT], u32x4 w, int kt, int xcol, int HT, int B,
                                         const uint16_t *xs, const uint16_t *xs_lo, int rstride) {
    constexpr int NA = NAcc<PRO>::n;
    constexpr bool HASLO = PRO != PRO_PAIR;
    const int lane = threadIdx.x & 63, j = lane & 15, g = lane >> 4;
    const u32x4 zero = u32x4{0u, 0u, 0u, 0u};
#pragma unroll
    for (int bt = 0; bt < NBT; ++bt) {
        // columns b >= B multiply row 0 again: MFMA columns are independent
        // and every epilogue drops them
        const int b = bt * 16 + j;
        const int xo = (b < B ? b : 0) * rstride + xcol + g * 8;
        const u32x4 bop = *(const u32x4 *)(xs + xo);
        const u32x4 bol = HASLO ? *(const u32x4 *)(xs_lo + xo) : zero;
        if (NA == 2) {
            // MTP: tiles below H/32 act on RMSNorm(h_b), the rest on RMSNorm(E[b])
            const bool hi_half = kt >= HT;
            const u32x4 w0 = hi_half ? zero : w, w1 = hi_half ? w : zero;
            acc[0][bt] = mfma16(w0, bop, acc[0][bt]);
            acc[0][bt] = mfma16(w0, bol, acc[0][bt]);
            acc[NA - 1][bt] = mfma16(w1, bop, acc[NA - 1][bt]);
            acc[NA - 1][bt] = mfma16(w1, bol, acc[NA - 1][bt]);
        } else {
            acc[0][bt] = mfma16(w, bop, acc[0][bt]);
            if (HASLO) acc[0][bt] = mfma16(w, bol, acc[0][bt]);
        }
    }
}

// RoPE inputs of one strip, requested ahead of its epilogue (the batch-1
// GEMV's strip groups): the position of each column's sequence and the
// cos / sin quadruple of this lane's rows.
template <int NBT>
struct QkvPre {
    int pos[NBT];
    float4 cs[NBT], sn[NBT];
};

// The RoPE rotation index of v = 0 for lane group g in a q or k strip.
__device__ __forceinline__ int rope_jr(int strip, int qs, int hs, int g) {
    const int sidx = strip < qs ? strip : strip - qs;
    return 8 * (sidx % hs) + 4 * (g & 1);
}

// Fused epilogues, one wave per strip (lanes (j, g) hold rows row0 + v of
// column b = 16 bt + j): bias or residual add with sum-of-squares parts,
// SwiGLU, RoPE + KV append, logits + argmax key.  pre (EPI_QKV): the RoPE
// inputs already in registers; NULL: read here.
template <int NBT, int EPI>
__device__ __forceinline__ void gemv_epilogue(const GemvParams &p, f32x4 (&fin)[NBT], const f32x4 (&resid)[NBT],
                                              int strip, bool lead, const QkvPre<NBT> *pre = nullptr) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int j = lane & 15, g = lane >> 4;
    const int nstrips = p.N >> 4;
    const int B = p.B;
    const int row0 = strip * 16 + 4 * g;
    if (EPI == EPI_LOGITS) {
        // every wave reaches here; waves without a strip contribute key 0
        __shared__ uint64_t s_best[kNW][kMaxB];
#pragma unroll
        for (int bt = 0; bt < NBT; ++bt) {
            const int b = bt * 16 + j;
            const bool ok = lead && b < B;
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
                if (g == 0) s_best[wave][b] = key;
            }
        }
        if (p.best) {
            __syncthreads();
            if (threadIdx.x < B) {
                uint64_t m = 0;
#pragma unroll
                for (int w = 0; w < kNW; ++w) m = s_best[w][threadIdx.x] > m ? s_best[w][threadIdx.x] : m;
                if (m) atomicMax((unsigned long long *)(p.best + threadIdx.x), (unsigned long long)m);
            }
        }
        return;
    }
    if (!lead) return;
    if (EPI == EPI_STORE || EPI == EPI_RESID) {
#pragma unroll
        for (int bt = 0; bt < NBT; ++bt) {
            const int b = bt * 16 + j;
            const bool ok = b < B;
            f32x4 val = fin[bt];
            if (EPI == EPI_RESID) val += resid[bt];
            else if (p.bias) val += *(const f32x4 *)(p.bias + row0);
            if (ok) *(f32x4 *)(p.out + (int64_t)b * p.N + row0) = val;
            float sq = val[0] * val[0] + val[1] * val[1] + val[2] * val[2] + val[3] * val[3];
            sq = col_sum(sq);
            if (ok && g == 0 && p.ss_out) p.ss_out[b * nstrips + strip] = sq;
        }
    } else if (EPI == EPI_SILU) {
#pragma unroll
        for (int bt = 0; bt < NBT; ++bt) {
            const int b = bt * 16 + j;
            if (b < B) {
                f32x4 w;
#pragma unroll
                for (int v = 0; v < 4; ++v) w[v] = silu_f(fin[bt][v]);
                *(f32x4 *)(p.act + (int64_t)b * p.N + row0) = w;
            }
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
        const int qs = p.n_q * hs, kvs = p.n_kv * hs;
#pragma unroll
        for (int bt = 0; bt < NBT; ++bt) {
            const int b = bt * 16 + j;
            f32x4 other;
#pragma unroll
            for (int v = 0; v < 4; ++v) other[v] = __shfl_xor(fin[bt][v], 32);
            if (b >= B) continue;
            const int pos = pre ? pre->pos[bt] : p.pos[b];
            if (strip < qs + kvs) {
                const bool isq = strip < qs;
                const int sidx = isq ? strip : strip - qs;
                const int head = sidx / hs, t = sidx - head * hs;
                const int jr = 8 * t + 4 * (g & 1);         // rotation index of v = 0
                const int dim0 = (g < 2) ? jr : (d >> 1) + jr;
                const float4 cs = pre ? pre->cs[bt] : *(const float4 *)(p.rope_cos + (int64_t)pos * (d >> 1) + jr);
                const float4 sn = pre ? pre->sn[bt] : *(const float4 *)(p.rope_sin + (int64_t)pos * (d >> 1) + jr);
                const float c4[4] = {cs.x, cs.y, cs.z, cs.w}, s4[4] = {sn.x, sn.y, sn.z, sn.w};
                float r[4];
#pragma unroll
                for (int v = 0; v < 4; ++v)
                    r[v] = (g < 2) ? fin[bt][v] * c4[v] - other[v] * s4[v] : fin[bt][v] * c4[v] + other[v] * s4[v];
                if (isq) {
                    *(f32x4 *)(p.q + ((int64_t)b * p.n_q + head) * d + dim0) = f32x4{r[0], r[1], r[2], r[3]};
                } else {
                    u32x2 w;
                    w[0] = pack_bf2(r[0], r[1]);
                    w[1] = pack_bf2(r[2], r[3]);
                    *(u32x2 *)(p.kc + (int64_t)b * p.kv_bstride + (int64_t)head * p.lmax_pad * d +
                               tiled_index(pos, dim0, d)) = w;
                }
            } else {
                const int r0 = (strip - qs - kvs) * 16 + 4 * g;
                const int kvh = r0 / d, dim = r0 - kvh * d;
                uint16_t *dst = p.vc + (int64_t)b * p.kv_bstride +
                                ((int64_t)(kvh * (p.lmax_pad >> 5) + (pos >> 5)) * d + dim) * 32 + vslot(pos & 31);
#pragma unroll
                for (int v = 0; v < 4; ++v) dst[v * 32] = (uint16_t)f2bf(fin[bt][v]);
            }
        }
    }
}

template <int NBT, int KS, int PRO, int EPI, int U>
__global__ __launch_bounds__(512) void k_gemv(GemvParams p) {
    // U: k-tiles per wave per load batch (two batches in flight).  Every
    // wave's slices of X fit in LDS at once (wave-private staging).  A
    // workgroup takes strip groups blockIdx.x, blockIdx.x + gridDim.x, ...:
    // X is staged once and the weight stream runs on across strip groups,
    // each group ending in its reduction and epilogue.
    static_assert(KS > 1, "the strip reduction orders the RMSNorm scalars");
    constexpr int SPW = kNW / KS;          // strips per strip group
    constexpr int NA = NAcc<PRO>::n;
    constexpr bool HASLO = PRO != PRO_PAIR;   // gathered embeddings are exact in bf16
    extern __shared__ __align__(16) uint16_t xs[];
    __shared__ float sc0[kMaxB], sc1[kMaxB];

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int j = lane & 15, g = lane >> 4;
    const int nstrips = p.N >> 4;
    const int ks = wave % KS;              // k-split index inside the strip
    const int slot = wave / KS;            // strip of this wave inside a group
    const int G = (nstrips + SPW - 1) / SPW;
    const int ngrp = (G - 1 - (int)blockIdx.x) / (int)gridDim.x + 1;   // groups of this workgroup
    const int KT = p.K >> 5, HT = p.H >> 5;
    const int B = p.B;
    const u32x4 zero = u32x4{0u, 0u, 0u, 0u};
    // LDS: X hi planes, X lo planes, then the reduction buffer
    const int nmax = (KT + KS - 1) / KS;                  // k-tiles of a wave per strip (uniform)
    const int n = (KT - ks + KS - 1) / KS;                // ... of which real for this wave
    const int nb = (nmax + U - 1) / U;                    // load batches per strip
    const int rstride = nmax * 32 + 8;                    // row stride of a wave's X slices
    const int xplane = kNW * B * rstride;                 // elements per plane set
    f32x4 *red = (f32x4 *)(xs + (HASLO ? 2 : 1) * xplane);   // [kNW][NBT][64] f32x4
    auto strip_of = [&](int r) { return ((int)blockIdx.x + r * (int)gridDim.x) * SPW + slot; };
    const int strip0 = strip_of(0);
    const int row00 = strip0 * 16 + 4 * g;

    f32x4 acc[NA][NBT];
#pragma unroll
    for (int a = 0; a < NA; ++a)
#pragma unroll
        for (int bt = 0; bt < NBT; ++bt) acc[a][bt] = f32x4{0.f, 0.f, 0.f, 0.f};

    // EPI_QKV: the RoPE inputs of group r's strip, requested while the group
    // streams (the positions once, with the prologue), so that its epilogue
    // waits on nothing
    QkvPre<NBT> qpre;
    auto rope_fetch = [&](int r) {
        const int strip = strip_of(r);
        const int hs = p.d >> 4, qs = p.n_q * hs, kvs = p.n_kv * hs;
        const bool rot = strip < qs + kvs;
        const int jr = rope_jr(rot ? strip : 0, qs, hs, g);
#pragma unroll
        for (int bt = 0; bt < NBT; ++bt) {
            const int64_t at = (int64_t)qpre.pos[bt] * (p.d >> 1) + jr;
            qpre.cs[bt] = *(const float4 *)(p.rope_cos + (rot ? at : 0));
            qpre.sn[bt] = *(const float4 *)(p.rope_sin + (rot ? at : 0));
        }
    };

    // Strip group r ends: KS partial sums reduced in wave order, RMSNorm
    // scalar, epilogue; the accumulators restart at zero.
    Pro<NBT, PRO, EPI> pr;
    auto finish = [&](int r) {
        f32x4 fin[NBT];
#pragma unroll
        for (int bt = 0; bt < NBT; ++bt) {
            f32x4 v = acc[0][bt];
            if (NA == 2) {
                const int b = bt * 16 + j;
                const float s0 = b < B ? sc0[b] : 0.f, s1 = b < B ? sc1[b] : 0.f;
                v = v * s0 + acc[NA - 1][bt] * s1;
            }
            fin[bt] = v;
        }
#pragma unroll
        for (int a = 0; a < NA; ++a)
#pragma unroll
            for (int bt = 0; bt < NBT; ++bt) acc[a][bt] = f32x4{0.f, 0.f, 0.f, 0.f};
        __syncthreads();
#pragma unroll
        for (int bt = 0; bt < NBT; ++bt) red[(wave * NBT + bt) * 64 + lane] = fin[bt];
        __syncthreads();
        if (ks == 0) {
#pragma unroll
            for (int bt = 0; bt < NBT; ++bt) {
#pragma unroll
                for (int w = 1; w < KS; ++w) fin[bt] += red[((wave + w) * NBT + bt) * 64 + lane];
            }
        }
        if (PRO == PRO_NORM || PRO == PRO_CAT) {
#pragma unroll
            for (int bt = 0; bt < NBT; ++bt) {
                const int b = bt * 16 + j;
                fin[bt] *= (b < B ? sc0[b] : 0.f);
            }
        }
        const int strip = strip_of(r);
        const bool lead = ks == 0 && strip < nstrips;
        f32x4 resid[NBT];
#pragma unroll
        for (int bt = 0; bt < NBT; ++bt) {
            resid[bt] = pr.resid[bt];
            if (EPI == EPI_RESID && r > 0) {   // later groups read their residual rows here
                const int b = bt * 16 + j;
                f32x4 v = *(const f32x4 *)(p.out + ((lead && b < B) ? (int64_t)b * p.N + strip * 16 + 4 * g : 0));
                // (opaque, so that the two sources stay two values: merged into
                // one load through a chosen pointer they would put pr in scratch)
                asm volatile("" : "+v"(v));
                resid[bt] = v;
            }
        }
        if constexpr (EPI == EPI_QKV) {
            gemv_epilogue<NBT, EPI>(p, fin, resid, strip, lead, &qpre);
            if (r + 1 < ngrp) rope_fetch(r + 1);   // the next group's, ahead of its stream's end
        } else {
            gemv_epilogue<NBT, EPI>(p, fin, resid, strip, lead);
        }
    };

    // ---- wave-private X, then one pipelined pass over every group's tiles ----
    // Batch q covers tiles i = U (q % nb) + u of strip group q / nb, at k-tile
    // ks + KS i.  Loads are unconditional (tiles past a strip's end or past
    // the last group read the matrix's first line and are multiplied as
    // zero), so every batch keeps a fixed load count and the waits before
    // each batch cover exactly that batch.
    const int nq = ngrp * nb;
    ChunkMap cm{true, nmax * 4, B * nmax * 4, ks, KS, KT, rstride};
    uint16_t *xh = xs + wave * B * rstride, *xl = xh + xplane;
    // 1. prologue / epilogue inputs, before any weights
    pro_load<NBT, PRO, EPI>(p, pr, ks == 0 && strip0 < nstrips, row00, cm, 0);
    if constexpr (EPI == EPI_QKV) {
#pragma unroll
        for (int bt = 0; bt < NBT; ++bt) {
            const int b = bt * 16 + j;
            qpre.pos[bt] = p.pos[b < B ? b : 0];
        }
    }
    // 2. two batches of weights
    u32x4 ra[U], rb[U];
    auto wptr = [&](int q, int u) -> const u32x4 * {
        const int r = q / nb, i = (q - r * nb) * U + u;
        const int strip = strip_of(r);
        const bool ok = q < nq && i < n && strip < nstrips;
        return (const u32x4 *)(ok ? p.W + ((int64_t)strip * KT + ks + KS * i) * 512 + lane * 8 : p.W);
    };
#pragma unroll
    for (int u = 0; u < U; ++u) ra[u] = __builtin_nontemporal_load(wptr(0, u));
#pragma unroll
    for (int u = 0; u < U; ++u) rb[u] = __builtin_nontemporal_load(wptr(1, u));
    // keep the prologue arithmetic (and its waits) after the weight loads
    __builtin_amdgcn_sched_barrier(0);
    // 3. scalars and this wave's slices of X; the MTP scales its halves
    //    before the reduction, so it waits for every wave's scalars
    pro_finish<NBT, PRO, EPI>(p, pr, cm, 0, xh, xl, sc0, sc1);
    if constexpr (EPI == EPI_QKV) rope_fetch(0);
    if (PRO == PRO_MTP) __syncthreads();
    // 4. stream: consume one batch while the next is in flight
    auto mma_batch = [&](const u32x4 (&R)[U], int q) {
        const int r = q / nb, i0 = (q - r * nb) * U;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int i = i0 + u;
            const bool ok = q < nq && i < n;
            tile_mma<NBT, PRO>(acc, ok ? R[u] : zero, ok ? ks + KS * i : 0, ok ? 32 * i : 0, HT, B, xh, xl, rstride);
        }
        if (q < nq && i0 + U >= nmax) finish(r);
    };
    // the last pair is peeled so that no load is left in flight at the end
    int q = 0;
    for (; q + 2 < nq; q += 2) {
        mma_batch(ra, q);
#pragma unroll
        for (int u = 0; u < U; ++u) ra[u] = __builtin_nontemporal_load(wptr(q + 2, u));
        mma_batch(rb, q + 1);
#pragma unroll
        for (int u = 0; u < U; ++u) rb[u] = __builtin_nontemporal_load(wptr(q + 3, u));
    }
    mma_batch(ra, q);
    mma_batch(rb, q + 1);
}

// ---------------------------------------------------------------------------
// The vocabulary head at larger batches.  k_xprep: one workgroup per row b
// writes X[b] = the GEMV input with its RMSNorm scale applied, split into
// bf16 hi / lo planes.  k_gemv_wide: a workgroup owns 128 weight rows (one
// 16-row strip per wave) over the whole K; chunks of X (all B rows, hi and
// lo) pass through LDS once per workgroup and are shared by its eight waves.
// Weights stream one chunk ahead of the chunk being multiplied.  The head
// never splits K: its argmax epilogue is workgroup-wide.
template <int PRO>
__global__ __launch_bounds__(256) void k_xprep(GemvParams p) {
    // workgroup (b, segment): columns [2048 seg, 2048 seg + 2048) of row b
    const int b = blockIdx.x / p.xseg, seg = blockIdx.x - b * p.xseg;
    const int K = p.K, H = p.H;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    __shared__ float s_part[2][4];
    float sc0 = 1.f, sc1 = 1.f;
    if (PRO == PRO_NORM || PRO == PRO_MTP || PRO == PRO_CAT) {
        // the row's sum of squares (and the MTP embedding row's), 8 values
        // requested per thread per step
        const int Kn = PRO == PRO_NORM ? K : H;
        const float *xr = p.x + (int64_t)b * Kn;
        float a = 0.f, e = 0.f;
#pragma unroll 4
        for (int k0 = threadIdx.x * 8; k0 < Kn; k0 += 256 * 8) {
            const float4 u0 = *(const float4 *)(xr + k0), u1 = *(const float4 *)(xr + k0 + 4);
            a += u0.x * u0.x + u0.y * u0.y + u0.z * u0.z + u0.w * u0.w;
            a += u1.x * u1.x + u1.y * u1.y + u1.z * u1.z + u1.w * u1.w;
        }
        if (PRO == PRO_CAT) {
            const float *x2 = p.x2 + (int64_t)b * H;
            for (int k0 = threadIdx.x * 8; k0 < H; k0 += 256 * 8) {
                const float4 u0 = *(const float4 *)(x2 + k0), u1 = *(const float4 *)(x2 + k0 + 4);
                a += u0.x * u0.x + u0.y * u0.y + u0.z * u0.z + u0.w * u0.w;
                a += u1.x * u1.x + u1.y * u1.y + u1.z * u1.z + u1.w * u1.w;
            }
        }
        if (PRO == PRO_MTP) {
            const int tok = clamp_id(argmax_key_id(p.tokkey[b]), p.vocab);
#pragma unroll 4
            for (int k0 = threadIdx.x * 8; k0 < H; k0 += 256 * 8) {
                const u32x4 w = *(const u32x4 *)(p.embed + tiled_index(tok, k0, H));
#pragma unroll
                for (int i = 0; i < 4; ++i) e += bf_lo(w[i]) * bf_lo(w[i]) + bf_hi(w[i]) * bf_hi(w[i]);
            }
        }
        a = wave_sum(a);
        e = wave_sum(e);
        if (lane == 0) {
            s_part[0][wave] = a;
            s_part[1][wave] = e;
        }
        __syncthreads();
        sc0 = rsqrtf((s_part[0][0] + s_part[0][1] + s_part[0][2] + s_part[0][3]) / (float)(PRO == PRO_CAT ? K : Kn) +
                     p.eps);
        sc1 = rsqrtf((s_part[1][0] + s_part[1][1] + s_part[1][2] + s_part[1][3]) / (float)H + p.eps);
    }
    {
        const int k = seg * 2048 + threadIdx.x * 8;
        if (k >= K) return;
        XSrc sx;
        load_src<PRO>(p, b, k, sx);
        u32x4 vh, vl;
        if (PRO == PRO_PAIR) {
            vh = sx.e;
            vl = u32x4{0u, 0u, 0u, 0u};
        } else {
            float f[8];
            if (PRO == PRO_F32) {
                f[0] = sx.a0.x; f[1] = sx.a0.y; f[2] = sx.a0.z; f[3] = sx.a0.w;
                f[4] = sx.a1.x; f[5] = sx.a1.y; f[6] = sx.a1.z; f[7] = sx.a1.w;
            } else if (PRO == PRO_NORM || PRO == PRO_CAT || k < H) {
                f[0] = sx.a0.x * sx.g0.x; f[1] = sx.a0.y * sx.g0.y; f[2] = sx.a0.z * sx.g0.z; f[3] = sx.a0.w * sx.g0.w;
                f[4] = sx.a1.x * sx.g1.x; f[5] = sx.a1.y * sx.g1.y; f[6] = sx.a1.z * sx.g1.z; f[7] = sx.a1.w * sx.g1.w;
#pragma unroll
                for (int i = 0; i < 8; ++i) f[i] *= sc0;
            } else {
                f[0] = bf_lo(sx.e[0]) * sx.g0.x; f[1] = bf_hi(sx.e[0]) * sx.g0.y; f[2] = bf_lo(sx.e[1]) * sx.g0.z;
                f[3] = bf_hi(sx.e[1]) * sx.g0.w; f[4] = bf_lo(sx.e[2]) * sx.g1.x; f[5] = bf_hi(sx.e[2]) * sx.g1.y;
                f[6] = bf_lo(sx.e[3]) * sx.g1.z; f[7] = bf_hi(sx.e[3]) * sx.g1.w;
#pragma unroll
                for (int i = 0; i < 8; ++i) f[i] *= sc1;
            }
            split8(f, vh, vl);
        }
        *(u32x4 *)(p.xh + (int64_t)b * K + k) = vh;
        *(u32x4 *)(p.xl + (int64_t)b * K + k) = vl;
    }
}

template <int NBT, int EPI>
__global__ __launch_bounds__(512) void k_gemv_wide(GemvParams p) {
    constexpr int CK = wide_chunk(NBT);    // k-tiles per X chunk
    constexpr int RS = CK * 32 + 8;        // LDS row stride (elements) of a chunk plane
    constexpr int XU = 2 * NBT * CK / 8;   // 16-byte X units per thread per chunk (2 B CK 4 / 512)
    extern __shared__ __align__(16) uint16_t xsm[];   // [2 buffers][2 planes][B][RS]
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int j = lane & 15, g = lane >> 4;
    const int nstrips = p.N >> 4;
    const int strip = blockIdx.x * kNW + wave;
    const bool sok = strip < nstrips;
    const int KT = p.K >> 5, K = p.K, B = p.B;
    const int c0 = 0, c1 = (KT + CK - 1) / CK;   // chunks over the whole K
    const int nch = c1 - c0;
    const uint16_t *wp = p.W + (int64_t)(sok ? strip : 0) * KT * 512 + lane * 8;
    const u32x4 zero = u32x4{0u, 0u, 0u, 0u};
    const int bufsz = 2 * B * RS;
    // X unit u of a chunk: plane, row, 8-column group
    const int units = 2 * B * (CK * 4);
    auto x_src = [&](int c, int r) -> const u32x4 * {
        int u = threadIdx.x + r * 512;
        u = u < units ? u : 0;
        const int plane = u / (B * CK * 4), rem = u - plane * B * CK * 4;
        const int b = rem / (CK * 4), c8 = rem - b * CK * 4;
        int col = (c0 + c) * CK * 32 + c8 * 8;
        col = (c0 + c < c1 && col < K) ? col : 0;
        return (const u32x4 *)((plane ? p.xl : p.xh) + (int64_t)b * K + col);
    };
    // units past the chunk land in a scratch line after the two buffers, so
    // the store (like the load) is unconditional
    auto x_put = [&](int buf, int r, u32x4 v) {
        const int u = threadIdx.x + r * 512;
        const int uc = u < units ? u : 0;
        const int plane = uc / (B * CK * 4), rem = uc - plane * B * CK * 4;
        const int b = rem / (CK * 4), c8 = rem - b * CK * 4;
        const int off = u < units ? buf * bufsz + plane * B * RS + b * RS + c8 * 8 : 2 * bufsz;
        *(u32x4 *)(xsm + off) = v;
    };
    // weight tile t of chunk c (tiles past K or past this range read the first line)
    auto w_src = [&](int c, int t) -> const u32x4 * {
        const int kt = (c0 + c) * CK + t;
        return (const u32x4 *)((c0 + c < c1 && kt < KT) ? wp + (int64_t)kt * 512 : p.W);
    };
    f32x4 acc[NBT];
#pragma unroll
    for (int bt = 0; bt < NBT; ++bt) acc[bt] = f32x4{0.f, 0.f, 0.f, 0.f};
    auto consume = [&](int buf, int c, const u32x4 (&w)[CK]) {
        const uint16_t *xh = xsm + buf * bufsz, *xl = xh + B * RS;
#pragma unroll
        for (int t = 0; t < CK; ++t) {
            const int kt = (c0 + c) * CK + t;
            const u32x4 wt = kt < KT ? w[t] : zero;
#pragma unroll
            for (int bt = 0; bt < NBT; ++bt) {
                const int b = bt * 16 + j;
                const int xo = (b < B ? b : 0) * RS + t * 32 + g * 8;
                u32x4 bh = *(const u32x4 *)(xh + xo), bl = *(const u32x4 *)(xl + xo);
                bh = b < B ? bh : zero;
                bl = b < B ? bl : zero;
                acc[bt] = mfma16(wt, bh, acc[bt]);
                acc[bt] = mfma16(wt, bl, acc[bt]);
            }
        }
    };
    f32x4 resid[NBT];
#pragma unroll
    for (int bt = 0; bt < NBT; ++bt) {
        const int b = bt * 16 + j;
        resid[bt] = f32x4{0.f, 0.f, 0.f, 0.f};
        if (EPI == EPI_RESID)
            resid[bt] = *(const f32x4 *)(p.out + ((sok && b < B) ? (int64_t)b * p.N + strip * 16 + 4 * g : 0));
    }
    // chunk c: X regs loaded one chunk ahead and written to LDS buffer c % 2
    // just before the barrier that opens chunk c; weights two chunks deep
    u32x4 xr[XU], wa[CK], wb[CK];
#pragma unroll
    for (int r = 0; r < XU; ++r) xr[r] = *x_src(0, r);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int t = 0; t < CK; ++t) wa[t] = __builtin_nontemporal_load(w_src(0, t));
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int r = 0; r < XU; ++r) x_put(0, r, xr[r]);
    __syncthreads();
#pragma unroll
    for (int r = 0; r < XU; ++r) xr[r] = *x_src(1, r);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int t = 0; t < CK; ++t) wb[t] = __builtin_nontemporal_load(w_src(1, t));
    __builtin_amdgcn_sched_barrier(0);
    for (int c = 0; c < nch; c += 2) {
        consume(0, c, wa);
#pragma unroll
        for (int r = 0; r < XU; ++r) x_put(1, r, xr[r]);
        __syncthreads();
#pragma unroll
        for (int r = 0; r < XU; ++r) xr[r] = *x_src(c + 2, r);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int t = 0; t < CK; ++t) wa[t] = __builtin_nontemporal_load(w_src(c + 2, t));
        __builtin_amdgcn_sched_barrier(0);
        if (c + 1 < nch) consume(1, c + 1, wb);
#pragma unroll
        for (int r = 0; r < XU; ++r) x_put(0, r, xr[r]);
        __syncthreads();
#pragma unroll
        for (int r = 0; r < XU; ++r) xr[r] = *x_src(c + 3, r);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int t = 0; t < CK; ++t) wb[t] = __builtin_nontemporal_load(w_src(c + 3, t));
        __builtin_amdgcn_sched_barrier(0);
    }
    f32x4 fin[NBT];
#pragma unroll
    for (int bt = 0; bt < NBT; ++bt) fin[bt] = acc[bt];
    gemv_epilogue<NBT, EPI>(p, fin, resid, strip, sok);
}

// ---------------------------------------------------------------------------
// Batches whose X does not fit wave-private (k_gemv_kr).  K is cut into
// ksplit ranges of krt k-tiles; workgroup w works on range w % ksplit,
// stages that range's slice of X (all B rows, hi and lo) in LDS once, and
// its eight waves then stream whole 16-row strips of the range, each wave on
// its own strips: after the staging there is no barrier and no cross-wave
// reduction.  A wave's tiles over all its strips form one stream in batches
// of U, two batches in flight, loads unconditional (tiles past the stream
// read the matrix's first line and are multiplied as zero).  With one range
// the wave runs the fused epilogue per strip; otherwise it writes the
// strip's partial sums (RMSNorm scale applied) and k_gemv_fin adds the
// ranges in range order.
// Where the k-range partial sums of range r, strip `strip`, sequence b start
// (16 rows follow).  Above 16 sequences the partials that k_gemv_fin reads
// by strip are [range][strip][B][16], so that one strip of every sequence is
// one contiguous block (whole cache lines for the partials' writer and
// reader; 4B at batch 32: 9.68 -> 9.55 ms per pair step); QKV's, which the
// decode attention reads by sequence, and those of smaller batches (where
// the blocked form measured slightly slower) are [range][B][N].
template <int NBT, int EPI>
__device__ __forceinline__ int64_t part_index(int r, int strip, int b, int B, int nstrips) {
    if (EPI == EPI_QKV || NBT == 1) return ((int64_t)r * B + b) * ((int64_t)nstrips * 16) + strip * 16;
    return (((int64_t)r * nstrips + strip) * B + b) * 16;
}
constexpr int kKrLdsBytes = 128 * 1024;      // X slice budget of a k-range workgroup (one per CU)
constexpr int kKrChunks = 8;                 // X chunks per thread: B * k-tiles * 4 <= 8 * 512
template <int PRO>   // the MTP's chunks hold both halves' sources, and PRO_CAT keeps two sets of
                     // RMSNorm parts, so fewer fit in registers
struct KrChunks { static constexpr int n = (PRO == PRO_MTP || PRO == PRO_CAT) ? 6 : kKrChunks; };
// the k-range choice's model (host side): KB per microsecond the chip
// streams and one wave streams (two 8 KB batches in flight), and the cost of a
// finishing launch in microseconds
constexpr double kKrChipRate = 6000.0, kKrWaveRate = 5.0, kKrFinUs = 5.0;
template <int NBT, int PRO, int EPI, int U>
__global__ __launch_bounds__(512) void k_gemv_kr(GemvParams p) {
    constexpr int NA = NAcc<PRO>::n;
    extern __shared__ __align__(16) uint16_t xs[];
    __shared__ float sc0[kMaxB], sc1[kMaxB];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int j = lane & 15, g = lane >> 4;
    const int nstrips = p.N >> 4;
    const int KT = p.K >> 5, HT = p.H >> 5, B = p.B;
    const int R = p.ksplit;
    const int r = (int)blockIdx.x % R;                         // this workgroup's k-range
    const int wr = ((int)gridDim.x - r + R - 1) / R;          // workgroups on range r
    const int wid = ((int)blockIdx.x / R) * kNW + wave;       // this wave among the range's waves
    const int nwr = wr * kNW;
    const int kt0 = r * p.krt;
    const int nt = min(p.krt, KT - kt0);                       // k-tiles of this range
    const int rstride = p.krt * 32 + 8;
    uint16_t *xh = xs, *xl = xs + B * rstride;
    const u32x4 zero = u32x4{0u, 0u, 0u, 0u};
    const int ns = wid < nstrips ? (nstrips - 1 - wid) / nwr + 1 : 0;   // strips wid, wid + nwr, ...
    const int nb = (nt + U - 1) / U;                          // batches per strip (the last one padded)
    const int nq = ns * nb;
    // tile u of batch q: strip q / nb, k-tile U (q % nb) + u of the range
    auto wptr = [&](int q, int u) -> const u32x4 * {
        const int sidx = q / nb, i = (q - sidx * nb) * U + u;
        const int strip = wid + sidx * nwr;
        return (const u32x4 *)(q < nq && i < nt ? p.W + ((int64_t)strip * KT + kt0 + i) * 512 + lane * 8 : p.W);
    };
    // 1. the RMSNorm inputs, then the whole X slice (at most KC 8-column
    //    chunks per thread), requested at once
    constexpr bool NORM = PRO == PRO_NORM || PRO == PRO_MTP || PRO == PRO_CAT;
    const int per_row = nt * 4, count = B * per_row;
    const int col0 = kt0 * 32;
    constexpr int KC = KrChunks<PRO>::n;
    constexpr int RPW = 2 * NBT;
    float ssv[RPW][4], ssv2[PRO == PRO_CAT ? RPW : 1][4];
    if (NORM) {
#pragma unroll
        for (int rr = 0; rr < RPW; ++rr)
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                const int b = wave + rr * kNW, i = lane + 64 * t;
                ssv[rr][t] = p.ss[(b < B && i < p.nss) ? b * p.nss + i : 0];
                if (PRO == PRO_CAT) ssv2[rr][t] = p.ss2[(b < B && i < p.nss) ? b * p.nss + i : 0];
            }
    }
    XSrc src[KC];
#pragma unroll
    for (int c = 0; c < KC; ++c) {
        int idx = threadIdx.x + c * (kNW * 64);
        idx = idx < count ? idx : 0;
        const int b = idx / per_row;
        load_src<PRO>(p, b, col0 + ((idx - b * per_row) << 3), src[c]);
    }
    // up to 16 sequences the weight batches go out right behind the X slice's
    // requests, before it arrives (9B at batch 8: 5.79 -> 5.76 ms per pair step)
    u32x4 ra[U], rb[U];
    auto issue_w = [&]() {
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int u = 0; u < U; ++u) ra[u] = __builtin_nontemporal_load(wptr(0, u));
#pragma unroll
        for (int u = 0; u < U; ++u) rb[u] = __builtin_nontemporal_load(wptr(1, u));
        __builtin_amdgcn_sched_barrier(0);
    };
    if constexpr (NBT == 1) issue_w();
    // 2. the slice into LDS (shared by the eight waves), the RMSNorm scalars
#pragma unroll
    for (int c = 0; c < KC; ++c) {
        const int idx = threadIdx.x + c * (kNW * 64);
        if (idx < count) {
            const int b = idx / per_row, k = (idx - b * per_row) << 3;
            u32x4 vh, vl;
            make_chunk<PRO>(p, col0 + k, src[c], vh, vl);
            *(u32x4 *)(xh + b * rstride + k) = vh;
            if (PRO != PRO_PAIR) *(u32x4 *)(xl + b * rstride + k) = vl;
        }
    }
    // above 16 sequences the weight batches go out once this workgroup's X
    // has arrived, before the scalars and the barrier (issued before it
    // arrives they queue ahead of its 64-128 KB slice: 9.39 instead of
    // 9.28 ms per pair step at 4B, batch 32)
    if constexpr (NBT != 1) issue_w();
    if (NORM) {
#pragma unroll
        for (int rr = 0; rr < RPW; ++rr) {
            const int b = wave + rr * kNW;
            float a = 0.f;
#pragma unroll
            for (int t = 0; t < 4; ++t) a += (lane + 64 * t < p.nss) ? ssv[rr][t] : 0.f;
            if (PRO == PRO_CAT) {
#pragma unroll
                for (int t = 0; t < 4; ++t) a += (lane + 64 * t < p.nss) ? ssv2[rr][t] : 0.f;
            }
            a = wave_sum_dpp(a);
            if (b < B && lane == 0) sc0[b] = rsqrtf(a / (float)(PRO == PRO_MTP ? p.H : p.K) + p.eps);
        }
    }
    if (PRO == PRO_MTP) {   // RMSNorm scale of E[tok] (a short row)
        for (int b = wave; b < B; b += kNW) {
            const int tok = clamp_id(argmax_key_id(p.tokkey[b]), p.vocab);
            float e2 = 0.f;
            for (int k = lane * 8; k < p.H; k += 512) {
                const u32x4 w = *(const u32x4 *)(p.embed + tiled_index(tok, k, p.H));
#pragma unroll
                for (int i = 0; i < 4; ++i) e2 += bf_lo(w[i]) * bf_lo(w[i]) + bf_hi(w[i]) * bf_hi(w[i]);
            }
            e2 = wave_sum_dpp(e2);
            if (lane == 0) sc1[b] = rsqrtf(e2 / (float)p.H + p.eps);
        }
    }
    __syncthreads();

    f32x4 acc[NA][NBT];
#pragma unroll
    for (int a = 0; a < NA; ++a)
#pragma unroll
        for (int bt = 0; bt < NBT; ++bt) acc[a][bt] = f32x4{0.f, 0.f, 0.f, 0.f};
    auto finish = [&](int sidx) {
        const int strip = wid + sidx * nwr;
        f32x4 fin[NBT];
#pragma unroll
        for (int bt = 0; bt < NBT; ++bt) {
            const int b = bt * 16 + j;
            const float s0 = b < B ? sc0[b] : 0.f;
            f32x4 v = acc[0][bt];
            if (NA == 2) v = v * s0 + acc[NA - 1][bt] * (b < B ? sc1[b] : 0.f);
            else if (PRO == PRO_NORM || PRO == PRO_CAT) v *= s0;
            fin[bt] = v;
        }
#pragma unroll
        for (int a = 0; a < NA; ++a)
#pragma unroll
            for (int bt = 0; bt < NBT; ++bt) acc[a][bt] = f32x4{0.f, 0.f, 0.f, 0.f};
        if (R == 1) {
            f32x4 resid[NBT];
#pragma unroll
            for (int bt = 0; bt < NBT; ++bt) {
                const int b = bt * 16 + j;
                resid[bt] = f32x4{0.f, 0.f, 0.f, 0.f};
                if (EPI == EPI_RESID)
                    resid[bt] = *(const f32x4 *)(p.out + (b < B ? (int64_t)b * p.N + strip * 16 + 4 * g : 0));
            }
            gemv_epilogue<NBT, EPI>(p, fin, resid, strip, true);
        } else {
#pragma unroll
            for (int bt = 0; bt < NBT; ++bt) {
                const int b = bt * 16 + j;
                if (b < B) *(f32x4 *)(p.part + part_index<NBT, EPI>(r, strip, b, B, nstrips) + 4 * g) = fin[bt];
            }
        }
    };
    auto consume = [&](const u32x4 (&Rg)[U], int q) {
        const int sidx = q / nb, i0 = (q - sidx * nb) * U;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int i = i0 + u;
            const bool ok = q < nq && i < nt;
            tile_mma<NBT, PRO>(acc, ok ? Rg[u] : zero, ok ? kt0 + i : 0, ok ? 32 * i : 0, HT, B, xh, xl, rstride);
        }
        if (q < nq && i0 + U >= nt) finish(sidx);
    };
    // 3. stream; the last pair of batches is peeled so no load is left in flight
    int q = 0;
    for (; q + 2 < nq; q += 2) {
        consume(ra, q);
#pragma unroll
        for (int u = 0; u < U; ++u) ra[u] = __builtin_nontemporal_load(wptr(q + 2, u));
        consume(rb, q + 1);
#pragma unroll
        for (int u = 0; u < U; ++u) rb[u] = __builtin_nontemporal_load(wptr(q + 3, u));
    }
    consume(ra, q);
    consume(rb, q + 1);
}

// Sum of the k-range partials in range order, then the fused epilogue.
template <int NBT, int EPI>
// One wave per strip (the vocabulary head never splits K, so the logits
// epilogue's workgroup-wide argmax is not needed here).
__global__ __launch_bounds__(64) void k_gemv_fin(GemvParams p) {
    const int lane = threadIdx.x & 63;
    const int j = lane & 15, g = lane >> 4;
    const int nstrips = p.N >> 4;
    const int strip = blockIdx.x;
    const bool sok = strip < nstrips;
    const int B = p.B;
    const int row0 = (sok ? strip : 0) * 16 + 4 * g;
    f32x4 fin[NBT], resid[NBT];
#pragma unroll
    for (int bt = 0; bt < NBT; ++bt) {
        const int b = bt * 16 + j;
        const int bc = b < B ? b : 0;
        resid[bt] = f32x4{0.f, 0.f, 0.f, 0.f};
        if (EPI == EPI_RESID) resid[bt] = *(const f32x4 *)(p.out + (int64_t)bc * p.N + row0);
        // request 16 ranges at a time, add them in range order
        f32x4 a = f32x4{0.f, 0.f, 0.f, 0.f};
        for (int k0 = 0; k0 < p.ksplit; k0 += 16) {
            f32x4 v[16];
#pragma unroll
            for (int u = 0; u < 16; ++u) {
                const int k = min(k0 + u, p.ksplit - 1);
                v[u] = *(const f32x4 *)(p.part + part_index<NBT, EPI>(k, sok ? strip : 0, bc, B, nstrips) + 4 * g);
            }
#pragma unroll
            for (int u = 0; u < 16; ++u)
                if (k0 + u < p.ksplit) a += v[u];
        }
        fin[bt] = a;
    }
    gemv_epilogue<NBT, EPI>(p, fin, resid, strip, sok);
}

template <int NBT, int KS, int PRO, int EPI, int U>
static void launch_multi(GemvParams &q, hipStream_t s);

template <int NBT, int KS, int PRO, int EPI, int U>
static void launch_t(const GemvParams &p, hipStream_t s) {
    GemvParams q = p;
    const int KT = q.K >> 5;
    constexpr int planes = PRO == PRO_PAIR ? 1 : 2;
    constexpr int SPW = kNW / KS;
    int grid = ((q.N >> 4) + SPW - 1) / SPW;
    const int red = kNW * NBT * 64 * 16;
    // wave-private X when every wave's slices fit
    const int nmax = (KT + KS - 1) / KS;
    const int lds_one = planes * kNW * q.B * (nmax * 32 + 8) * 2 + red;
    constexpr int budget = (EPI == EPI_RESID || EPI == EPI_SWIGLU) ? kGemvOneLdsBytesWide : kGemvOneLdsBytes;
    if (NBT <= 2 && lds_one <= budget) {   // (never fits beyond 32 columns)
        if (q.wg_cap > 0 && grid > q.wg_cap) grid = q.wg_cap;
        if (g_gemv_timing.pending) {
            hipExtLaunchKernelGGL((k_gemv<NBT, KS, PRO, EPI, U>), dim3(grid), dim3(kNW * 64), lds_one, s,
                                  g_gemv_timing.start, g_gemv_timing.stop, 0, q);
            g_gemv_timing.pending = false;
        } else {
            hipLaunchKernelGGL((k_gemv<NBT, KS, PRO, EPI, U>), dim3(grid), dim3(kNW * 64), lds_one, s, q);
        }
        return;
    }
    // the other paths launch several kernels: the events bracket them
    const bool timed = g_gemv_timing.pending;
    g_gemv_timing.pending = false;
    if (timed) hipEventRecord(g_gemv_timing.start, s);
    launch_multi<NBT, KS, PRO, EPI, U>(q, s);
    if (timed) hipEventRecord(g_gemv_timing.stop, s);
}

template <int NBT, int KS, int PRO, int EPI, int U>
static void launch_multi(GemvParams &q, hipStream_t s) {
    const int KT = q.K >> 5;
    // below the vocabulary head: k-ranges whose X slices fit
    if constexpr (EPI != EPI_LOGITS) {
        // k-tiles per range: the X slice (hi + lo bf16) within the LDS budget
        // and the per-thread chunk count, and enough ranges x strips for the
        // streaming waves
        int kmax = kKrLdsBytes / (2 * 2 * q.B * 32);
        const int krt_c = KrChunks<PRO>::n * kNW * 64 / (4 * q.B);
        kmax = (kmax < krt_c ? kmax : krt_c) / 4 * 4;
        // the split with the shortest estimated time: ranges of nearly equal
        // length (a multiple of 4 k-tiles), every range on the same number of
        // workgroups, each wave streaming its strips in rounds; the stream
        // takes the longer of the matrix at the chip's bandwidth and one wave's
        // share at a wave's rate (at most the bandwidth split over the active
        // waves); more than one range adds the finishing launch and the
        // partial sums it writes and reads
        const int S = q.N >> 4, wg = q.wg_cap > 0 ? q.wg_cap : 256;
        const double total = (double)S * KT;                      // 1 KB tiles
        int R = 0, krt = 0;
        double best = 1e30;
        for (int kt = 4; kt <= kmax; kt += 4) {
            const int r0 = (KT + kt - 1) / kt;
            const int ke = ((KT + r0 - 1) / r0 + 3) / 4 * 4;     // even ranges
            if (ke > kmax) continue;
            const int r = (KT + ke - 1) / ke;
            const int nwr = (wg / r > 0 ? wg / r : 1) * kNW;
            const double active = (double)std::min(S, nwr) * r;
            const double rate = std::min(kKrWaveRate, kKrChipRate / active);
            double t = std::max(total / kKrChipRate, (double)((S + nwr - 1) / nwr) * ke / rate);
            if (r > 1) t += kKrFinUs + 2.0 * r * q.B * q.N * 4 / 1024.0 / kKrChipRate;
            if (t < best - 1e-9) best = t, R = r, krt = ke;
        }
        const bool partials = R > 1 && (int64_t)R * q.B * q.N <= q.part_cap;
        if (R > 0 && (R == 1 || partials)) {
            q.ksplit = R;
            q.krt = krt;
            const int lds_kr = 2 * q.B * (krt * 32 + 8) * 2;
            const int grid_kr = ((q.wg_cap > 0 ? q.wg_cap : 256) / R) * R;   // whole rounds of ranges
            hipLaunchKernelGGL((k_gemv_kr<NBT, PRO, EPI, 8>), dim3(grid_kr > R ? grid_kr : R), dim3(kNW * 64),
                               lds_kr, s, q);
            if (EPI == EPI_QKV && R > 1 && R <= kAttnFusedRanges && q.deferred) *q.deferred = R;   // the attention finishes it
            else if (R > 1) hipLaunchKernelGGL((k_gemv_fin<NBT, EPI>), dim3(q.N >> 4), dim3(64), 0, s, q);
            return;
        }
    }
    // the vocabulary head (and any matrix whose partials would not fit the
    // workspace): X planes, then 128-row workgroups over the whole K
    q.xseg = (q.K + 2047) / 2048;
    hipLaunchKernelGGL((k_xprep<PRO>), dim3(q.B * q.xseg), dim3(256), 0, s, q);
    const int rtiles = ((q.N >> 4) + kNW - 1) / kNW;
    const int lds_w = 2 * 2 * q.B * (wide_chunk(NBT) * 32 + 8) * 2 + 16;
    hipLaunchKernelGGL((k_gemv_wide<NBT, EPI>), dim3(rtiles), dim3(kNW * 64), lds_w, s, q);
}

// Batch size U: two batches of U tiles per wave are in flight.  Five when a
// wave's tile count is a multiple of ten (K = 2560 with an eight-way split:
// no padding tiles), four otherwise.
template <int NBT, int KS, int PRO, int EPI>
static void launch_u(const GemvParams &p, hipStream_t s) {
    const int n = ((p.K >> 5) + KS - 1) / KS;
    if (n % 10 == 0) launch_t<NBT, KS, PRO, EPI, 5>(p, s);
    else launch_t<NBT, KS, PRO, EPI, 4>(p, s);
}

template <int KS, int PRO, int EPI>
static void launch_nbt(const GemvParams &p, hipStream_t s) {
    if (p.B <= 16) launch_u<1, KS, PRO, EPI>(p, s);
    else if (p.B <= 32) launch_u<2, KS, PRO, EPI>(p, s);
    else if (p.B <= 48) launch_u<3, KS, PRO, EPI>(p, s);
    else launch_u<4, KS, PRO, EPI>(p, s);
}

int gemv_num_groups(int N) { return N >> 4; }

// One instantiation per (prologue, epilogue) pair the decode step uses.
// Waves per strip (the K split), from a sweep on MI355X at batch 1: the LM
// head (151936 rows) splits K in four, every other matrix in eight.  Any
// other pair launches nothing and returns -1.
int launch_gemv(const GemvParams &p, int pro, int epi, hipStream_t s) {
    if (pro == PRO_PAIR && epi == EPI_STORE) launch_nbt<8, PRO_PAIR, EPI_STORE>(p, s);
    else if (pro == PRO_NORM && epi == EPI_QKV) launch_nbt<8, PRO_NORM, EPI_QKV>(p, s);
    else if (pro == PRO_F32 && epi == EPI_RESID) launch_nbt<8, PRO_F32, EPI_RESID>(p, s);
    else if (pro == PRO_NORM && epi == EPI_SWIGLU) launch_nbt<8, PRO_NORM, EPI_SWIGLU>(p, s);
    else if (pro == PRO_NORM && epi == EPI_LOGITS) launch_nbt<4, PRO_NORM, EPI_LOGITS>(p, s);
    else if (pro == PRO_MTP && epi == EPI_STORE) launch_nbt<8, PRO_MTP, EPI_STORE>(p, s);
    else if (pro == PRO_NORM && epi == EPI_STORE) launch_nbt<8, PRO_NORM, EPI_STORE>(p, s);
    else if (pro == PRO_PAIR && epi == EPI_SILU) launch_nbt<8, PRO_PAIR, EPI_SILU>(p, s);
    else if (pro == PRO_CAT && epi == EPI_SILU) launch_nbt<8, PRO_CAT, EPI_SILU>(p, s);
    else return -1;
    return 0;
}

}  // namespace pipo
