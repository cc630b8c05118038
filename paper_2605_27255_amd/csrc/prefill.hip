// Compressed-prompt prefill: the pair step batched over a chunk of latent
// positions of every sequence.  Activations that feed an MFMA GEMM are kept
// in the 16x32 tiled bf16 layout, as two planes hi and lo (x ~= hi + lo,
// about 16 significant bits), so that both GEMM operands move as contiguous
// 1 KB tiles (weights straight into registers, activations through LDS).
#include "device_common.h"
#include "kernels.h"

namespace pipo {

__device__ __forceinline__ float silu_p(float u) { return u / (1.0f + __expf(-u)); }

// ---- pair gather: X_in[m] = [E[a]; E[b]] for latent c0 + i of sequence b ----
__global__ void k_gather_pairs(const int32_t *tokens, const uint16_t *embed, int H, int V, int pad_id,
                               PrefillGeom g, uint16_t *xin) {
    const int cpr = (2 * H) >> 3;
    const int64_t total = (int64_t)g.B * g.mpad * cpr;
    for (int64_t idx = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; idx < total;
         idx += (int64_t)gridDim.x * blockDim.x) {
        const int m = (int)(idx / cpr);
        const int k = (int)(idx - (int64_t)m * cpr) << 3;
        const int b = m / g.mpad, i = m - b * g.mpad;
        int row = pad_id;
        if (i < g.clen) {   // rows past a sequence's prompt (ragged batch) hold (PAD, PAD)
            const int t = 2 * (g.c0 + i) + (k < H ? 0 : 1);
            row = t < seq_tokens(g, b) ? clamp_id(tokens[(int64_t)b * g.n_tok + t], V) : pad_id;
        }
        const u32x4 v = *(const u32x4 *)(embed + tiled_index(row, k < H ? k : k - H, H));
        *(u32x4 *)(xin + tiled_index(m, k, 2 * H)) = v;
    }
}

void launch_gather_pairs(const int32_t *tokens, const uint16_t *embed, int H, int V, int pad_id,
                         const PrefillGeom &g, uint16_t *xin, hipStream_t s) {
    const int64_t total = (int64_t)g.B * g.mpad * ((2 * H) >> 3);
    int grid = (int)((total + 255) / 256);
    grid = grid > 65536 ? 65536 : grid;
    hipLaunchKernelGGL(k_gather_pairs, dim3(grid), dim3(256), 0, s, tokens, embed, H, V, pad_id, g, xin);
}

// ---- MLP compressor's skip path: x[m] = E[a] + E[b] for latent c0 + i -------
__global__ void k_gather_pair_sum(const int32_t *tokens, const uint16_t *embed, int H, int V, int pad_id,
                                  PrefillGeom g, float *x) {
    const int cpr = H >> 3;
    const int64_t total = (int64_t)g.B * g.mpad * cpr;
    for (int64_t idx = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; idx < total;
         idx += (int64_t)gridDim.x * blockDim.x) {
        const int m = (int)(idx / cpr);
        const int k = (int)(idx - (int64_t)m * cpr) << 3;
        const int b = m / g.mpad, i = m - b * g.mpad;
        int ra = pad_id, rb = pad_id;
        if (i < g.clen) {
            const int t = 2 * (g.c0 + i), nb = seq_tokens(g, b);
            ra = t < nb ? clamp_id(tokens[(int64_t)b * g.n_tok + t], V) : pad_id;
            rb = t + 1 < nb ? clamp_id(tokens[(int64_t)b * g.n_tok + t + 1], V) : pad_id;
        }
        const u32x4 va = *(const u32x4 *)(embed + tiled_index(ra, k, H));
        const u32x4 vb = *(const u32x4 *)(embed + tiled_index(rb, k, H));
        float4 *dst = (float4 *)(x + (int64_t)m * H + k);
        dst[0] = make_float4(bf_lo(va[0]) + bf_lo(vb[0]), bf_hi(va[0]) + bf_hi(vb[0]),
                             bf_lo(va[1]) + bf_lo(vb[1]), bf_hi(va[1]) + bf_hi(vb[1]));
        dst[1] = make_float4(bf_lo(va[2]) + bf_lo(vb[2]), bf_hi(va[2]) + bf_hi(vb[2]),
                             bf_lo(va[3]) + bf_lo(vb[3]), bf_hi(va[3]) + bf_hi(vb[3]));
    }
}

void launch_gather_pair_sum(const int32_t *tokens, const uint16_t *embed, int H, int V, int pad_id,
                            const PrefillGeom &g, float *x, hipStream_t s) {
    const int64_t total = (int64_t)g.B * g.mpad * (H >> 3);
    int grid = (int)((total + 255) / 256);
    grid = grid > 65536 ? 65536 : grid;
    hipLaunchKernelGGL(k_gather_pair_sum, dim3(grid), dim3(256), 0, s, tokens, embed, H, V, pad_id, g, x);
}

// ---- MTP layer inputs of the prompt's latents (one wave per row) -----------
// Row (b, i) = [RMSNorm(h_b; g_mh); RMSNorm(E[t]; g_me)] with t the prompt token
// after latent c0 + i's pair (PAD where there is none: the last latent, whose
// row is recomputed with the selected token once it is known), written as
// tiled hi / lo planes of width 2H.
__global__ __launch_bounds__(256) void k_mtp_rows(const float *xb, const int32_t *tokens, const uint16_t *embed,
                                                  const float *gh, const float *ge, int H, int V, int pad_id,
                                                  float eps, PrefillGeom g, int M, uint16_t *xh, uint16_t *xl) {
    const int lane = threadIdx.x & 63;
    const int m = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (m >= M) return;
    const int b = m / g.mpad, i = m - b * g.mpad;
    const int t = 2 * (g.c0 + i) + 2;
    const int tok = (i < g.clen && t < seq_tokens(g, b)) ? clamp_id(tokens[(int64_t)b * g.n_tok + t], V) : pad_id;
    const float *xr = xb + (int64_t)m * H;
    float a = 0.f, e = 0.f;
    for (int k = lane * 8; k < H; k += 512) {
        const float4 x0 = *(const float4 *)(xr + k), x1 = *(const float4 *)(xr + k + 4);
        a += x0.x * x0.x + x0.y * x0.y + x0.z * x0.z + x0.w * x0.w + x1.x * x1.x + x1.y * x1.y + x1.z * x1.z +
             x1.w * x1.w;
        const u32x4 w = *(const u32x4 *)(embed + tiled_index(tok, k, H));
#pragma unroll
        for (int q = 0; q < 4; ++q) e += bf_lo(w[q]) * bf_lo(w[q]) + bf_hi(w[q]) * bf_hi(w[q]);
    }
    a = wave_sum(a);
    e = wave_sum(e);
    const float s1 = rsqrtf(a / (float)H + eps), s2 = rsqrtf(e / (float)H + eps);
    for (int k = lane * 8; k < H; k += 512) {
        const float4 x0 = *(const float4 *)(xr + k), x1 = *(const float4 *)(xr + k + 4);
        const float4 g0 = *(const float4 *)(gh + k), g1 = *(const float4 *)(gh + k + 4);
        const float f[8] = {x0.x * s1 * g0.x, x0.y * s1 * g0.y, x0.z * s1 * g0.z, x0.w * s1 * g0.w,
                            x1.x * s1 * g1.x, x1.y * s1 * g1.y, x1.z * s1 * g1.z, x1.w * s1 * g1.w};
        u32x4 hi, lo;
        split8(f, hi, lo);
        const int64_t at = tiled_index(m, k, 2 * H);
        *(u32x4 *)(xh + at) = hi;
        *(u32x4 *)(xl + at) = lo;
        const u32x4 w = *(const u32x4 *)(embed + tiled_index(tok, k, H));
        const float4 e0 = *(const float4 *)(ge + k), e1 = *(const float4 *)(ge + k + 4);
        const float fe[8] = {bf_lo(w[0]) * s2 * e0.x, bf_hi(w[0]) * s2 * e0.y, bf_lo(w[1]) * s2 * e0.z,
                             bf_hi(w[1]) * s2 * e0.w, bf_lo(w[2]) * s2 * e1.x, bf_hi(w[2]) * s2 * e1.y,
                             bf_lo(w[3]) * s2 * e1.z, bf_hi(w[3]) * s2 * e1.w};
        split8(fe, hi, lo);
        const int64_t at2 = tiled_index(m, H + k, 2 * H);
        *(u32x4 *)(xh + at2) = hi;
        *(u32x4 *)(xl + at2) = lo;
    }
}

void launch_mtp_rows(const float *xb, const int32_t *tokens, const uint16_t *embed, const float *gh, const float *ge,
                     int H, int V, int pad_id, float eps, const PrefillGeom &g, int M, uint16_t *xh, uint16_t *xl,
                     hipStream_t s) {
    hipLaunchKernelGGL(k_mtp_rows, dim3((M + 3) / 4), dim3(256), 0, s, xb, tokens, embed, gh, ge, H, V, pad_id, eps,
                       g, M, xh, xl);
}

// ---- regular decoding: the prompt's tokens one per position, x = E[t] -----
// Row (b, i) of the chunk holds token c0 + i of sequence b (rows past the
// chunk hold E[pad_id]); fp32 residual rows [B * mpad][H].
__global__ void k_gather_tokens(const int32_t *tokens, const uint16_t *embed, int H, int V, int pad_id,
                                PrefillGeom g, float *x) {
    const int cpr = H >> 3;
    const int64_t total = (int64_t)g.B * g.mpad * cpr;
    for (int64_t idx = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; idx < total;
         idx += (int64_t)gridDim.x * blockDim.x) {
        const int m = (int)(idx / cpr);
        const int k = (int)(idx - (int64_t)m * cpr) << 3;
        const int b = m / g.mpad, i = m - b * g.mpad;
        const int t = g.c0 + i;
        const int row = (i < g.clen && t < seq_tokens(g, b)) ? clamp_id(tokens[(int64_t)b * g.n_tok + t], V) : pad_id;
        const u32x4 v = *(const u32x4 *)(embed + tiled_index(row, k, H));
        float4 *dst = (float4 *)(x + (int64_t)m * H + k);
        dst[0] = make_float4(bf_lo(v[0]), bf_hi(v[0]), bf_lo(v[1]), bf_hi(v[1]));
        dst[1] = make_float4(bf_lo(v[2]), bf_hi(v[2]), bf_lo(v[3]), bf_hi(v[3]));
    }
}

void launch_gather_tokens(const int32_t *tokens, const uint16_t *embed, int H, int V, int pad_id,
                          const PrefillGeom &g, float *x, hipStream_t s) {
    const int64_t total = (int64_t)g.B * g.mpad * (H >> 3);
    int grid = (int)((total + 255) / 256);
    grid = grid > 65536 ? 65536 : grid;
    hipLaunchKernelGGL(k_gather_tokens, dim3(grid), dim3(256), 0, s, tokens, embed, H, V, pad_id, g, x);
}

// ---- RMSNorm of fp32 rows into the tiled bf16 layout ----------------------
// One workgroup per 16-row tile row: wave w first forms the sums of squares
// of rows 4w..4w+3 (the four rows' loads interleaved), then writes every
// fourth 16x32 tile whole: lane l normalises row l mod 16, columns
// 8 (l / 16) .. + 7 of the tile, so each store instruction covers one
// contiguous 1 KB tile (full cache lines, no partial-line writes shared with
// other workgroups).
__global__ __launch_bounds__(256) void k_rmsnorm_tiled(const float *x, const float *gain, int H, float eps,
                                                       int M, uint16_t *xh, uint16_t *xl) {
    __shared__ float s_sc[16];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int r0 = blockIdx.x * 16;
    if (r0 >= M) return;
    {
        const float *xr = x + (int64_t)(r0 + 4 * wave) * H;
        float a[4] = {0.f, 0.f, 0.f, 0.f};
        for (int k = lane * 4; k < H; k += 256) {
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const float4 v = *(const float4 *)(xr + (int64_t)q * H + k);
                a[q] += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
            }
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const float t = wave_sum(a[q]);
            if (lane == 0) s_sc[4 * wave + q] = rsqrtf(t / (float)H + eps);
        }
    }
    __syncthreads();
    const int j = lane & 15, c = lane >> 4;
    const float sc = s_sc[j];
    const float *xr = x + (int64_t)(r0 + j) * H;
    const int KT = H >> 5;
    uint16_t *th = xh + (int64_t)(r0 >> 4) * KT * 512 + lane * 8;
    uint16_t *tl = xl + (int64_t)(r0 >> 4) * KT * 512 + lane * 8;
    for (int kt = wave; kt < KT; kt += 4) {
        const int k = kt * 32 + c * 8;
        const float4 x0 = *(const float4 *)(xr + k), x1 = *(const float4 *)(xr + k + 4);
        const float4 g0 = *(const float4 *)(gain + k), g1 = *(const float4 *)(gain + k + 4);
        const float f[8] = {x0.x * sc * g0.x, x0.y * sc * g0.y, x0.z * sc * g0.z, x0.w * sc * g0.w,
                            x1.x * sc * g1.x, x1.y * sc * g1.y, x1.z * sc * g1.z, x1.w * sc * g1.w};
        u32x4 hi, lo;
        split8(f, hi, lo);
        *(u32x4 *)(th + (int64_t)kt * 512) = hi;
        *(u32x4 *)(tl + (int64_t)kt * 512) = lo;
    }
}

void launch_rmsnorm_tiled(const float *x, const float *gain, int H, float eps, int M, uint16_t *xh,
                          uint16_t *xl, hipStream_t s) {
    // M is a multiple of 16 (chunk rows are padded to 32 per sequence)
    hipLaunchKernelGGL(k_rmsnorm_tiled, dim3((M + 15) / 16), dim3(256), 0, s, x, gain, H, eps, M, xh, xl);
}

// ---- MFMA GEMM  C^T[N][M] = W[N][K] X[M][K]^T, both operands tiled ---------
// Fused epilogue of one 16x16 accumulator fragment: lane (j, g) holds rows
// 16 strip + 4 g + v of token m.  Every lane takes part in the shuffles
// before any of them returns.
template <int EPI>
__device__ __forceinline__ void gemm_epi(const GemmParams &p, f32x4 val, int strip, int m) {
    const int lane = threadIdx.x & 63, g = lane >> 4;
    f32x4 other;
    if (EPI == EPI_SWIGLU || EPI == EPI_QKV) {
#pragma unroll
        for (int v = 0; v < 4; ++v) other[v] = __shfl_xor(val[v], 32);
    }
    if (strip >= (p.N >> 4) || m >= p.M) return;
    const int b = m / p.g.mpad, i = m - b * p.g.mpad;
    if (i >= p.g.clen) return;
    const int row0 = strip * 16 + 4 * g;
    if (EPI == EPI_STORE) {
        if (p.bias) val += *(const f32x4 *)(p.bias + row0);
        *(f32x4 *)(p.out + (int64_t)m * p.N + row0) = val;
    } else if (EPI == EPI_RESID) {
        f32x4 *o = (f32x4 *)(p.out + (int64_t)m * p.N + row0);
        *o = *o + val;
    } else if (EPI == EPI_SILU) {
        uint32_t h[4], l[4];
#pragma unroll
        for (int v = 0; v < 4; ++v) split_bf(silu_p(val[v]), h[v], l[v]);
        const int64_t at = tiled_index(m, row0, p.N);
        *(u32x2 *)(p.act_hi + at) = u32x2{h[0] | (h[1] << 16), h[2] | (h[3] << 16)};
        *(u32x2 *)(p.act_lo + at) = u32x2{l[0] | (l[1] << 16), l[2] | (l[3] << 16)};
    } else if (EPI == EPI_SWIGLU) {
        if (g < 2) {
            uint32_t h[4], l[4];
#pragma unroll
            for (int v = 0; v < 4; ++v) split_bf(silu_p(val[v]) * other[v], h[v], l[v]);
            const int64_t at = tiled_index(m, strip * 8 + 4 * g, p.N >> 1);
            *(u32x2 *)(p.act_hi + at) = u32x2{h[0] | (h[1] << 16), h[2] | (h[3] << 16)};
            *(u32x2 *)(p.act_lo + at) = u32x2{l[0] | (l[1] << 16), l[2] | (l[3] << 16)};
        }
    } else if (EPI == EPI_QKV) {
        const int d = p.d, hs = d >> 4;
        const int qs = p.n_q * hs, ks = p.n_kv * hs;
        const int pos = p.g.c0 + i;
        if (strip < qs + ks) {
            const bool isq = strip < qs;
            const int sidx = isq ? strip : strip - qs;
            const int head = sidx / hs, t = sidx - head * hs;
            const int jr = 8 * t + 4 * (g & 1);
            const int dim0 = (g < 2) ? jr : (d >> 1) + jr;
            const float *cs = p.rope_cos + (int64_t)pos * (d >> 1) + jr;
            const float *sn = p.rope_sin + (int64_t)pos * (d >> 1) + jr;
            float r[4];
#pragma unroll
            for (int v = 0; v < 4; ++v)
                r[v] = (g < 2) ? val[v] * cs[v] - other[v] * sn[v] : val[v] * cs[v] + other[v] * sn[v];
            if (isq) {   // the query as a bf16 pair hi + lo (two planes)
                uint32_t h[4], l[4];
#pragma unroll
                for (int v = 0; v < 4; ++v) split_bf(r[v], h[v], l[v]);
                const int64_t at = (((int64_t)b * p.n_q + head) * p.g.mpad + i) * d + dim0;
                *(u32x2 *)(p.q + at) = u32x2{h[0] | (h[1] << 16), h[2] | (h[3] << 16)};
                *(u32x2 *)(p.q_lo + at) = u32x2{l[0] | (l[1] << 16), l[2] | (l[3] << 16)};
            } else {     // the key, stored in bf16 (the cache's format)
                u32x2 w;
                w[0] = pack_bf2(r[0], r[1]);
                w[1] = pack_bf2(r[2], r[3]);
                *(u32x2 *)(p.kc + (int64_t)b * p.kv_bstride + (int64_t)head * p.lmax_pad * d +
                           tiled_index(pos, dim0, d)) = w;
            }
        } else {
            const int r0 = (strip - qs - ks) * 16 + 4 * g;
            const int kvh = r0 / d, dim = r0 - kvh * d;
            uint16_t *dst = p.vc + (int64_t)b * p.kv_bstride +
                            ((int64_t)(kvh * (p.lmax_pad >> 5) + (pos >> 5)) * d + dim) * 32 + vslot(pos & 31);
#pragma unroll
            for (int v = 0; v < 4; ++v) dst[v * 32] = (uint16_t)f2bf(val[v]);
        }
    }
}

// ---- MFMA GEMM  C^T[N][M] = W[N][K] X[M][K]^T, both operands tiled ---------
// Workgroup tile 256 (or 320) weight rows x 64 tokens, four waves of 64 (80) x 64 (4 (5) x 4
// fragments).  A wave's 64 weight rows are its own, so their 1 KB tiles go
// from memory straight into its registers (one contiguous load per tile, no
// LDS); the token tiles (X hi and lo, 16 KB per 64-wide k step) are shared by
// the four waves through a double-buffered LDS stage.  One iteration covers
// two 32-wide k tiles; the next iteration's weights and X are requested
// before this one's MFMAs, and X is written to LDS after them.  MFMAs run the
// hi plane over all 16 accumulators, then the lo plane, so dependent MFMAs
// are 16 apart (and every accumulator sees hi, lo of one k tile before the
// next k tile).
// Workgroups are placed per XCD (workgroup i runs on XCD i % 8): each XCD
// takes a contiguous run of tiles in grouped order (8 weight tiles by every
// token tile), so the ~64 workgroups resident on one XCD cover about 8 x 8
// tiles and share their weight and token tiles in that XCD's L2.
constexpr int kWdToks = 64, kWdGroup = 8;   // tokens per workgroup tile; weight tiles per XCD group

__device__ __forceinline__ bool wd_tile(int id, int nbn, int nbm, int &bn, int &bm) {
    const int T = nbn * nbm;
    const int chunk = (T + 7) / 8;
    const int u = (id & 7) * chunk + (id >> 3);
    if (u >= T) return false;
    const int gsz = kWdGroup * nbm;
    const int grp = u / gsz, r = u - grp * gsz;
    const int first = grp * kWdGroup;
    const int gs = min(kWdGroup, nbn - first);
    bn = first + r % gs;
    bm = r / gs;
    return true;
}

template <int EPI, bool HASLO, int SW>   // SW: 16-row weight strips per wave (tile of 64 SW rows)
__global__ __launch_bounds__(256) void k_gemm_wd(GemmParams p) {
    constexpr int NP = HASLO ? 2 : 1;
    constexpr int XT = NP * 2 * 4;                            // X tiles per stage: plane x k-tile x token strip
    constexpr int XC = XT / 4;                                // 16-byte X chunks per thread per stage
    extern __shared__ __align__(16) uint16_t lds[];           // [2][XT][512]
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int j = lane & 15;
    constexpr int ROWS = 64 * SW;
    const int nbn = (p.N + ROWS - 1) / ROWS, nbm = (p.M + kWdToks - 1) / kWdToks;
    int bn, bm;
    if (!wd_tile(blockIdx.x, nbn, nbm, bn, bm)) return;
    if (p.g.ntok) {   // a ragged batch: a token tile wholly past its sequence's last position holds only PAD rows
        const int m0 = bm * kWdToks, sb = m0 / p.g.mpad;   // (mpad is a multiple of the tile there)
        if (p.g.c0 + (m0 - sb * p.g.mpad) >= (p.g.ntok[sb] + p.g.tok_per_pos - 1) / p.g.tok_per_pos) return;
    }
    const int KT = p.K >> 5;
    const int NI = (KT + 1) >> 1;                              // iterations of two k tiles
    const int NS = p.N >> 4, MS = p.M >> 4;

    // this wave's SW weight strips (padding strips read strip 0, masked later)
    const uint16_t *wsrc[SW];
#pragma unroll
    for (int si = 0; si < SW; ++si) {
        int strip = bn * 4 * SW + wave * SW + si;
        strip = strip < NS ? strip : 0;
        wsrc[si] = p.W + (int64_t)strip * KT * 512 + lane * 8;
    }
    // X chunks of this thread: c = tid + 256 r, tile c / 64 = (plane, kk, ms)
    const uint16_t *xsrc[XC];
#pragma unroll
    for (int r = 0; r < XC; ++r) {
        const int c = tid + 256 * r, t = c >> 6, within = c & 63;
        const int plane = t >> 3, kk = (t >> 2) & 1, ms = t & 3;
        int strip = bm * 4 + ms;
        strip = strip < MS ? strip : 0;
        xsrc[r] = (plane ? p.Xlo : p.X) + ((int64_t)strip * KT + kk) * 512 + within * 8;
    }
    // k tiles past the end re-read the last one (their products are skipped)
    auto kclamp = [&](int kt) { return kt < KT ? kt : KT - 1; };
    auto load_w = [&](int it, u32x4 (&w)[2][SW]) {
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
#pragma unroll
            for (int si = 0; si < SW; ++si)
                w[kk][si] = *(const u32x4 *)(wsrc[si] + (int64_t)kclamp(2 * it + kk) * 512);
    };
    auto load_x = [&](int it, u32x4 (&x)[XC]) {
#pragma unroll
        for (int r = 0; r < XC; ++r) {
            const int kk = ((tid + 256 * r) >> 8) & 1;
            const int kt = kclamp(2 * it + kk) - kk;           // xsrc already holds the kk offset
            x[r] = *(const u32x4 *)(xsrc[r] + (int64_t)kt * 512);
        }
    };
    auto store_x = [&](int buf, const u32x4 (&x)[XC]) {
#pragma unroll
        for (int r = 0; r < XC; ++r) *(u32x4 *)(&lds[(buf * XT * 64 + tid + 256 * r) * 8]) = x[r];
    };

    f32x4 acc[SW][4];
#pragma unroll
    for (int a = 0; a < SW; ++a)
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[a][c] = f32x4{0.f, 0.f, 0.f, 0.f};

    auto mma = [&](int buf, int it, const u32x4 (&w)[2][SW]) {
        const uint16_t *L = lds + buf * XT * 512;
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
            if (kk == 1 && 2 * it + 1 >= KT) break;            // odd K: no second tile
            u32x4 bh[4], bl[4];
#pragma unroll
            for (int mi = 0; mi < 4; ++mi) {
                bh[mi] = *(const u32x4 *)(&L[((0 * 2 + kk) * 4 + mi) * 512 + lane * 8]);
                if (HASLO) bl[mi] = *(const u32x4 *)(&L[((1 * 2 + kk) * 4 + mi) * 512 + lane * 8]);
            }
#pragma unroll
            for (int si = 0; si < SW; ++si)
#pragma unroll
                for (int mi = 0; mi < 4; ++mi) acc[si][mi] = mfma16(w[kk][si], bh[mi], acc[si][mi]);
            if (HASLO) {
#pragma unroll
                for (int si = 0; si < SW; ++si)
#pragma unroll
                    for (int mi = 0; mi < 4; ++mi) acc[si][mi] = mfma16(w[kk][si], bl[mi], acc[si][mi]);
            }
        }
    };

    u32x4 wa[2][SW], wb[2][SW], xr[XC];
    load_x(0, xr);
    load_w(0, wa);
    store_x(0, xr);
    __syncthreads();
    // iteration it: request it + 1, multiply it, stage X of it + 1
    for (int it = 0; it < NI; it += 2) {
        load_x(it + 1, xr);
        load_w(it + 1, wb);
        mma(0, it, wa);
        store_x(1, xr);
        __syncthreads();
        if (it + 1 >= NI) break;
        load_x(it + 2, xr);
        load_w(it + 2, wa);
        mma(1, it + 1, wb);
        store_x(0, xr);
        __syncthreads();
    }

#pragma unroll
    for (int si = 0; si < SW; ++si)
#pragma unroll
        for (int mi = 0; mi < 4; ++mi)
            gemm_epi<EPI>(p, acc[si][mi], bn * 4 * SW + wave * SW + si, bm * kWdToks + mi * 16 + j);
}

// Tile height: 256 or 320 weight rows, whichever gives the busiest compute
// unit the fewest rows (workgroups are spread evenly over the 256 CUs, so a
// CU runs ceil(tiles / 256) of them): at N = 2560 the 256-row tile leaves
// 2.5 workgroups per CU (half the CUs run three), the 320-row tile two.
template <int EPI, bool HASLO>
static void launch_gemm_wd(const GemmParams &p, hipStream_t s) {
    const int nbm = (p.M + kWdToks - 1) / kWdToks;
    auto load = [&](int rows) {
        const int tiles = ((p.N + rows - 1) / rows) * nbm;
        return (int64_t)((tiles + 255) / 256) * rows;
    };
    const bool five = p.N % 320 == 0 && load(320) < load(256);
    const int nbn = five ? p.N / 320 : (p.N + 255) / 256;
    const int grid = 8 * ((nbn * nbm + 7) / 8);
    const size_t lds = 2 * (HASLO ? 16 : 8) * 1024;
    if (five) hipLaunchKernelGGL((k_gemm_wd<EPI, HASLO, 5>), dim3(grid), dim3(256), lds, s, p);
    else hipLaunchKernelGGL((k_gemm_wd<EPI, HASLO, 4>), dim3(grid), dim3(256), lds, s, p);
}

void launch_gemm(const GemmParams &p, hipStream_t s) {
    if (!p.Xlo) {   // the gathered embedding pairs are exact in bf16
        if (p.epi == EPI_SILU) launch_gemm_wd<EPI_SILU, false>(p, s);
        else launch_gemm_wd<EPI_STORE, false>(p, s);
        return;
    }
    switch (p.epi) {
        case EPI_STORE: launch_gemm_wd<EPI_STORE, true>(p, s); break;
        case EPI_RESID: launch_gemm_wd<EPI_RESID, true>(p, s); break;
        case EPI_SWIGLU: launch_gemm_wd<EPI_SWIGLU, true>(p, s); break;
        default: launch_gemm_wd<EPI_QKV, true>(p, s); break;
    }
}

// ---- causal grouped-query flash attention for a chunk of queries ----------
// One workgroup per (sequence, KV group, group of up to four query heads,
// 64-query block); eight waves, wave w computes head w % 4 for the block's
// 32-query half w / 4 (two 16-column MFMA tiles).  Keys and values of 64
// positions at a time are staged in LDS, shared by the workgroup's heads and
// halves and double-buffered: each stage is requested into registers two
// stages ahead (two register sets), and each lane writes the pieces it
// requested, widened from bf16 to fp16, into the other buffer half-way through
// the stage before (4B, 32768 latents: about 2% less attention time than one
// stage ahead).  Per stage the
// scores of all 64 keys are formed first (both query tiles), then one online-
// softmax update per query tile (the causal mask only on stages that reach the
// diagonal; stages wholly past a half's queries are skipped), so the row max /
// sum shuffles happen once per 64 keys, and the accumulators are rescaled only
// when the running max grows by more than 2^8.  Scores stay unscaled; the
// softmax scale 1/sqrt(d) (times log2 e) enters through one fma per score in
// the exponent, and the exponentials are the hardware exp2 (results below the
// normal range flush to zero, which the softmax weights can afford).
// Both products take fp16 operands: the query (its hi + lo pair summed and
// rounded once) and the probabilities carry 11 significant bits (against 8 for
// bf16), and K and V, stored as bf16, are widened to fp16 exactly for every
// value in fp16's normal range (|x| in [2^-14, 65504]; smaller values keep
// 2^-24 absolute precision; larger ones would overflow, a limit of this prefill
// kernel only).  One MFMA per product instead of a bf16 pair's two.
typedef __attribute__((ext_vector_type(8))) _Float16 f16x8;
typedef __attribute__((ext_vector_type(2))) _Float16 f16x2_t;
__device__ __forceinline__ uint32_t pack_f16x2(float lo, float hi) {
    const f16x2_t v = {(_Float16)lo, (_Float16)hi};
    return __builtin_bit_cast(uint32_t, v);
}
__device__ __forceinline__ f32x4 mfma16_f16(u32x4 a, u32x4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c, 0, 0,
                                                  0);
}

constexpr int kAQ = 64;         // queries per workgroup (two 32-query halves)
constexpr int kAK = 64;         // keys per LDS stage

template <int D>
__global__ __launch_bounds__(512, 1) void k_attn_prefill(AttnPrefillParams p) {
    constexpr int NC = D / 32, NT = D / 16;
    // two stage buffers, each the stage's K tiles (as in the cache) then its
    // V fragments in MFMA operand order; two named arrays, so that reading
    // one while the other fills is visibly independent
    __shared__ __align__(16) uint16_t kv_a[2 * kAK * D], kv_b[2 * kAK * D];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int j = lane & 15, g = lane >> 4;
    const int qpg = p.n_q / p.n_kv;
    const int nhg = (qpg + 3) / 4;               // head groups per KV group
    const int nqb = (p.g.clen + kAQ - 1) / kAQ;
    // heavy (late) query blocks first
    const int qblk = nqb - 1 - (int)(blockIdx.x % nqb);
    const int rest = blockIdx.x / nqb;
    const int hg = rest % nhg, bk = rest / nhg;
    const int b = bk / p.n_kv, kvh = bk - b * p.n_kv;
    const int hig = hg * 4 + (wave & 3);         // head index inside the KV group
    const bool active = hig < qpg;
    const int head = kvh * qpg + (active ? hig : 0);
    const int q0 = qblk * kAQ;                 // chunk-local first query of the workgroup
    const int qpos0 = p.g.c0 + q0;             // ... its absolute position
    const int q0w = q0 + 32 * (wave >> 2);     // this wave's first query (its half)
    const int qpos0w = p.g.c0 + q0w;
    const float scale = 1.4426950408889634f / sqrtf((float)D);
    // a ragged batch: a block wholly past this sequence's last position holds
    // only PAD rows, whose outputs nothing reads
    if (p.g.ntok && qpos0 >= (p.g.ntok[b] + p.g.tok_per_pos - 1) / p.g.tok_per_pos) return;

    u32x4 qb[2][NC];   // the query rows in fp16
#pragma unroll
    for (int ct = 0; ct < 2; ++ct)
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            const int row = min(q0w + 16 * ct + j, p.g.mpad - 1);   // rows past the chunk are never written
            const int64_t at = (((int64_t)b * p.n_q + head) * p.g.mpad + row) * D + 32 * c + 8 * g;
            const u32x4 h = *(const u32x4 *)(p.q + at), l = *(const u32x4 *)(p.q_lo + at);
#pragma unroll
            for (int i = 0; i < 4; ++i)
                qb[ct][c][i] = pack_f16x2(bf_lo(h[i]) + bf_lo(l[i]), bf_hi(h[i]) + bf_hi(l[i]));
        }

    const uint16_t *kbase = p.kc + (int64_t)b * p.kv_bstride + (int64_t)kvh * p.lmax_pad * D;
    const uint16_t *vbase = p.vc + (int64_t)b * p.kv_bstride + (int64_t)kvh * p.lmax_pad * D;

    f32x4 o[2][NT];
#pragma unroll
    for (int ct = 0; ct < 2; ++ct)
#pragma unroll
        for (int t = 0; t < NT; ++t) o[ct][t] = f32x4{0.f, 0.f, 0.f, 0.f};
    float m_run[2] = {-INFINITY, -INFINITY}, l_run[2] = {0.f, 0.f};

    const int kend = qpos0 + kAQ;              // keys [0, kend) may be visible
    // One 64-key stage: each lane requests 16 bytes of each of its wave's K
    // and V blocks into registers at the start of the previous stage, and
    // writes them widened to fp16 into the stage buffer half-way through it,
    // lane l at the block's base + 16 l (one LDS write per piece, against a
    // direct-to-LDS load plus a read and a write to convert in place): the K
    // tiles are 16 contiguous 1 KB blocks (D = 128) kept as they are; each 1 KB
    // V block (16 dims x 32 keys of a V tile) is read with its lanes permuted
    // so that lane l = 16 g + j holds dim j, keys 8 g .. 8 g + 7, the PV MFMA's
    // A operand, read back linearly.
    constexpr int KBW = D / 64;            // K (and V) blocks per wave per stage
    const int nstage = (kend + kAK - 1) / kAK;
    auto stage_issue = [&](u32x4 (&stg)[2 * KBW], int kb0) {
#pragma unroll
        for (int u = 0; u < KBW; ++u) {
            const int blk = wave * KBW + u;
            stg[u] = *(const u32x4 *)(kbase + (int64_t)kb0 * D + blk * 512 + lane * 8);
        }
#pragma unroll
        for (int u = 0; u < KBW; ++u) {
            const int vb = wave * KBW + u, h = vb / NT, t = vb - h * NT;
            stg[KBW + u] = *(const u32x4 *)(vbase + (int64_t)((kb0 >> 5) + h) * D * 32 + (16 * t + j) * 32 + 8 * g);
        }
    };
    // the pieces, bf16 -> fp16, into a stage buffer: K blocks as stored, V
    // blocks in MFMA operand order (each lane's piece at 16 bytes x lane)
    auto stage_f16 = [&](const u32x4 (&stg)[2 * KBW], uint16_t *buf) {
#pragma unroll
        for (int u = 0; u < 2 * KBW; ++u) {
            u32x4 h;
#pragma unroll
            for (int i = 0; i < 4; ++i) h[i] = pack_f16x2(bf_lo(stg[u][i]), bf_hi(stg[u][i]));
            *(u32x4 *)(buf + (u < KBW ? 0 : kAK * D) + (wave * KBW + (u % KBW)) * 512 + lane * 8) = h;
        }
    };
    // One 64-key stage: the scores of both 16-query tiles, the softmax of
    // tile 0, then the PV MFMAs of tile 0 with the softmax of tile 1 (VALU
    // that does not depend on them) issued between them, then tile 1's PV.
    // The scores are S^T over the four 16-key tiles; the softmax is one
    // online update per tile and stage; PV is O^T += V^T P^T.  The running
    // max only moves when some column's max grows by more than 2^8 (in exp2
    // units), so the accumulators are rarely rescaled and every exponent
    // stays at most 256; o / l at the end is the same quotient.  The rescale
    // decision (a branch) is taken before each overlapped phase.
    auto scores = [&](const uint16_t *ks, f32x4 (&s0)[4], f32x4 (&s1)[4]) {
#pragma unroll
        for (int tau = 0; tau < 4; ++tau) {
            u32x4 kf[NC];
#pragma unroll
            for (int c = 0; c < NC; ++c) kf[c] = *(const u32x4 *)(&ks[(tau * NC + c) * 512 + lane * 8]);
            s0[tau] = f32x4{0.f, 0.f, 0.f, 0.f};
            s1[tau] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int c = 0; c < NC; ++c) {
                s0[tau] = mfma16_f16(kf[c], qb[0][c], s0[tau]);
                s1[tau] = mfma16_f16(kf[c], qb[1][c], s1[tau]);
            }
        }
    };
    // masked scores (diagonal stages only), the column max and the rescale
    auto soft_max = [&](int ct, f32x4 (&sct)[4], int kb0, bool diag) {
        // keys past this column's query are masked
        const int lim = diag ? qpos0w + 16 * ct + j - kb0 - 4 * g : 64;
        float mx = -INFINITY;
#pragma unroll
        for (int tau = 0; tau < 4; ++tau)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                float sv = sct[tau][v];
                if (diag) sv = 16 * tau + v <= lim ? sv : -INFINITY;
                sct[tau][v] = sv;
                mx = fmaxf(mx, sv);
            }
        mx = col_max(mx);
        // a query row sees key 0 in the first stage, so the max is finite from then on
        const float m_cand = fmaxf(m_run[ct], mx * scale);
        if (__any(m_cand > m_run[ct] + 8.0f)) {
            const float alpha = __builtin_amdgcn_exp2f(m_run[ct] - m_cand);
            l_run[ct] *= alpha;
#pragma unroll
            for (int t = 0; t < NT; ++t) o[ct][t] *= alpha;
            m_run[ct] = m_cand;
        }
    };
    // probabilities, their sum and P^T in fp16
    auto soft_exp = [&](int ct, f32x4 (&sct)[4], u32x4 (&ph)[2]) {
        const float m_use = m_run[ct];
        float ps = 0.f;
#pragma unroll
        for (int tau = 0; tau < 4; ++tau)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const float e = __builtin_amdgcn_exp2f(fmaf(sct[tau][v], scale, -m_use));
                sct[tau][v] = e;
                ps += e;
            }
        l_run[ct] += col_sum(ps);
#pragma unroll
        for (int half = 0; half < 2; ++half)
#pragma unroll
            for (int i = 0; i < 4; ++i)
                ph[half][i] = pack_f16x2(sct[2 * half + (i >> 1)][2 * (i & 1)], sct[2 * half + (i >> 1)][2 * (i & 1) + 1]);
    };
    auto pv = [&](const uint16_t *vs, int ct, const u32x4 (&ph)[2]) {
#pragma unroll
        for (int half = 0; half < 2; ++half)
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                const u32x4 vf = *(const u32x4 *)(&vs[(half * NT + t) * 512 + lane * 8]);
                o[ct][t] = mfma16_f16(vf, ph[half], o[ct][t]);
            }
    };
    f32x4 s0[4], s1[4];
    u32x4 p0h[2], p1h[2];
    // Stage st + 2 is requested (into one register set) as stage st starts,
    // and stage st + 1, requested a stage earlier into the other set, lands in
    // the other buffer half-way through stage st: a full stage to arrive.
    auto stage = [&](int st, const uint16_t *cur, uint16_t *nxt, const u32x4 (&conv)[2 * KBW],
                     u32x4 (&iss)[2 * KBW]) {
        stage_issue(iss, min((st + 2) * kAK, p.lmax_pad - kAK));   // (a request past the end reads an unused stage)
        // the causal mask only where some key of the stage lies past some query
        // a wave skips stages wholly past its queries (the upper half's last
        // stage for the lower half) but still converts its share of the next
        const bool live = active && st * kAK <= qpos0w + 31;
        const bool diag = st * kAK + kAK - 1 > qpos0w;
        const uint16_t *vs = cur + kAK * D;
        if (live) {
            scores(cur, s0, s1);
            soft_max(0, s0, st * kAK, diag);
            soft_exp(0, s0, p0h);
        }
        // the next stage's pieces to fp16, between this stage's MFMA phases
        // (every wave, live or not, writes its share)
        stage_f16(conv, nxt);
        if (live) {
            soft_max(1, s1, st * kAK, diag);
            pv(vs, 0, p0h);
            soft_exp(1, s1, p1h);
            pv(vs, 1, p1h);
        }
        __syncthreads();
    };
    u32x4 sta[2 * KBW], stb[2 * KBW];   // this lane's 16-byte pieces of two coming stages
    stage_issue(sta, 0);
    stage_issue(stb, min(kAK, p.lmax_pad - kAK));
    stage_f16(sta, kv_a);
    __syncthreads();
    for (int st = 0; st < nstage; st += 2) {
        stage(st, kv_a, kv_b, stb, sta);
        if (st + 1 < nstage) stage(st + 1, kv_b, kv_a, sta, stb);
    }
    if (!active) return;
    const int qd = p.n_q * D;
#pragma unroll
    for (int ct = 0; ct < 2; ++ct) {
        const int i = q0w + 16 * ct + j;
        if (i >= p.g.clen) continue;
        const float inv = 1.0f / l_run[ct];
        const int64_t m = (int64_t)b * p.g.mpad + i;
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            uint32_t h[4], l[4];
#pragma unroll
            for (int v = 0; v < 4; ++v) split_bf(o[ct][t][v] * inv, h[v], l[v]);
            const int64_t at = tiled_index(m, head * D + 16 * t + 4 * g, qd);
            *(u32x2 *)(p.out_hi + at) = u32x2{h[0] | (h[1] << 16), h[2] | (h[3] << 16)};
            *(u32x2 *)(p.out_lo + at) = u32x2{l[0] | (l[1] << 16), l[2] | (l[3] << 16)};
        }
    }
}

void launch_attn_prefill(const AttnPrefillParams &p, hipStream_t s) {
    const int qpg = p.n_q / p.n_kv;
    const int nhg = (qpg + 3) / 4;
    const int nqb = (p.g.clen + kAQ - 1) / kAQ;
    const int grid = p.g.B * p.n_kv * nhg * nqb;
    const int threads = 512;   // eight waves stage K/V even when the group has fewer heads
    if (p.d == 128) hipLaunchKernelGGL(k_attn_prefill<128>, dim3(grid), dim3(threads), 0, s, p);
    else hipLaunchKernelGGL(k_attn_prefill<64>, dim3(grid), dim3(threads), 0, s, p);
}

// ---- last latent of each sequence into the decode residual buffer --------
// The last position's residual becomes the decode state x (with the
// sum-of-squares part of every 16-element strip, as the decode GEMVs read
// them); pos is set to that position, so the heads that follow run there and
// advance it, and the step counter restarts.
__global__ __launch_bounds__(256) void k_pick_last(const float *x, int H, PrefillGeom g, float *xdec,
                                                   float *ss, int32_t *pos, int32_t *step, int regular) {
    const int b = blockIdx.x;
    const int nb = seq_tokens(g, b);
    const int last = (regular ? nb : (nb + 1) / 2) - 1;   // the sequence's last position
    if (last < g.c0 || last >= g.c0 + g.clen) return;
    const float *xr = x + ((int64_t)b * g.mpad + last - g.c0) * H;
    for (int k = threadIdx.x; k < H; k += 256) xdec[(int64_t)b * H + k] = xr[k];
    for (int st = threadIdx.x; st < (H >> 4); st += 256) {
        float a = 0.f;
#pragma unroll
        for (int i = 0; i < 16; ++i) a += xr[16 * st + i] * xr[16 * st + i];
        ss[(int64_t)b * (H >> 4) + st] = a;
    }
    if (threadIdx.x == 0) {
        pos[b] = last;
        step[b] = 0;
    }
}

void launch_pick_last(const float *x, int H, const PrefillGeom &g, float *xdec, float *ss, int32_t *pos,
                      int32_t *step, int regular, hipStream_t s) {
    hipLaunchKernelGGL(k_pick_last, dim3(g.B), dim3(256), 0, s, x, H, g, xdec, ss, pos, step, regular);
}

}  // namespace pipo
