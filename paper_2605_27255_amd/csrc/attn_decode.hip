// Grouped-query flash-decode over the latent KV cache (one query position per
// sequence), split along the key axis.
//
// One wave per (sequence, KV group, split).  The group's query heads are the
// 16 columns of the MFMA tiles (unused columns are zero): scores are computed
// transposed, S^T[key][head] = K Q^T, 16 keys per tile, so each lane's
// accumulator holds one head; online softmax runs per column; the
// probabilities, held as (4g + v, 16 + 4g + v) for lane group g, are already
// the B operand of O^T[dim][head] += V^T P^T because the V cache stores each
// 32-key tile in that key order (see vslot in gemv.hip).  The query and the
// probabilities enter the MFMAs as bf16 pairs hi + lo (two MFMAs each), so
// only the bf16 KV cache itself limits the precision.  Per-split results
// (m, l, o) go to a partial buffer; a second kernel merges them per head in
// split order (the kernel boundary makes every split's partial visible).
#include "device_common.h"
#include "kernels.h"

namespace pipo {

template <int D>
__global__ __launch_bounds__(64) void k_attn_decode(AttnDecodeParams p) {
    constexpr int NC = D / 32;   // 32-wide d chunks (QK^T k-steps)
    constexpr int NT = D / 16;   // 16-wide d tiles (PV output tiles)
    const int lane = threadIdx.x, j = lane & 15, g = lane >> 4;
    const int S = p.splits;
    const int split = blockIdx.x % S;
    const int bk = blockIdx.x / S;               // b * n_kv + kvh
    const int b = bk / p.n_kv, kvh = bk - b * p.n_kv;
    const int qpg = p.n_q / p.n_kv;
    // splits own whole 32-key blocks: split s takes blocks [s*nb/S, (s+1)*nb/S)
    const int len = p.pos[b] + 1;
    const int nb = (len + 31) >> 5;
    const int k0 = ((split * nb) / S) * 32;
    const int k1 = min(len, (((split + 1) * nb) / S) * 32);
    const float scale = 1.4426950408889634f / sqrtf((float)D);

    // the query rows (clamped for unused columns, zeroed below) and the first
    // block are requested together, before any of them is waited for
    float4 qr[NC][2];
    {
        const int jq = j < qpg ? j : 0;
        const float4 *qp = (const float4 *)(p.q + ((int64_t)b * p.n_q + kvh * qpg + jq) * D + 8 * g);
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            qr[c][0] = qp[8 * c];
            qr[c][1] = qp[8 * c + 1];
        }
    }
    const uint16_t *kbase = p.kc + (int64_t)b * p.kv_bstride + (int64_t)kvh * p.lmax_pad * D;
    const uint16_t *vbase = p.vc + (int64_t)b * p.kv_bstride + (int64_t)kvh * p.lmax_pad * D;

    // K and V fragments of one 32-key block: two 16-key K tiles (one 1 KB
    // tile per 32 dims, stored in MFMA operand order, so each load is one
    // contiguous 1 KB read) and the 32-key V tile, 16 dims per output tile.
    // Every key is read once per step: nontemporal loads.
    u32x4 kf[2][2][NC], vf[2][NT];
    auto load_block = [&](int bsel, int kb) {
#pragma unroll
        for (int tau = 0; tau < 2; ++tau) {
            const uint16_t *kt = kbase + ((int64_t)((kb >> 4) + tau) * NC) * 512 + lane * 8;
#pragma unroll
            for (int c = 0; c < NC; ++c) kf[bsel][tau][c] = __builtin_nontemporal_load((const u32x4 *)(kt + c * 512));
        }
        const uint16_t *vt = vbase + (int64_t)(kb >> 5) * D * 32 + j * 32 + 8 * g;
#pragma unroll
        for (int t = 0; t < NT; ++t) vf[bsel][t] = __builtin_nontemporal_load((const u32x4 *)(vt + t * 16 * 32));
    };
    // blocks k0 + 32 i, i < nblk; loads past the end re-read the first block
    const int nblk = k0 < k1 ? (k1 - k0 + 31) >> 5 : 0;
    auto blk = [&](int i) { return i < nblk ? k0 + 32 * i : 0; };
    load_block(0, blk(0));
    load_block(1, blk(1));
    __builtin_amdgcn_sched_barrier(0);
    u32x4 qh[NC], ql[NC];
#pragma unroll
    for (int c = 0; c < NC; ++c) {
        const float f[8] = {qr[c][0].x, qr[c][0].y, qr[c][0].z, qr[c][0].w,
                            qr[c][1].x, qr[c][1].y, qr[c][1].z, qr[c][1].w};
        split8(f, qh[c], ql[c]);
        if (j >= qpg) {
            qh[c] = u32x4{0u, 0u, 0u, 0u};
            ql[c] = u32x4{0u, 0u, 0u, 0u};
        }
    }
    f32x4 o[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) o[t] = f32x4{0.f, 0.f, 0.f, 0.f};
    float m_run = -INFINITY, l_run = 0.f;
    auto block = [&](int bsel, int kb) {
        f32x4 st[2];
#pragma unroll
        for (int tau = 0; tau < 2; ++tau) {
            st[tau] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int c = 0; c < NC; ++c) {
                st[tau] = mfma16(kf[bsel][tau][c], qh[c], st[tau]);
                st[tau] = mfma16(kf[bsel][tau][c], ql[c], st[tau]);
            }
        }
        float mx = -INFINITY;
#pragma unroll
        for (int tau = 0; tau < 2; ++tau)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int key = kb + 16 * tau + 4 * g + v;
                const float sv = key < k1 ? st[tau][v] * scale : -INFINITY;
                st[tau][v] = sv;
                mx = fmaxf(mx, sv);
            }
        mx = col_max(mx);
        const float m_new = fmaxf(m_run, mx);
        const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
        float ps = 0.f;
#pragma unroll
        for (int tau = 0; tau < 2; ++tau)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const float e = __builtin_amdgcn_exp2f(st[tau][v] - m_new);
                st[tau][v] = e;
                ps += e;
            }
        l_run = l_run * alpha + col_sum(ps);
        m_run = m_new;
        const float pf[8] = {st[0][0], st[0][1], st[0][2], st[0][3], st[1][0], st[1][1], st[1][2], st[1][3]};
        u32x4 ph, pl;
        split8(pf, ph, pl);
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            o[t] *= alpha;
            o[t] = mfma16(vf[bsel][t], ph, o[t]);
            o[t] = mfma16(vf[bsel][t], pl, o[t]);
        }
    };
    // ping-pong over 32-key blocks: the next two blocks' loads are in flight
    // while one is computed, with a fixed load count per step
    int i = 0;
    for (; i + 2 < nblk; i += 2) {
        block(0, k0 + 32 * i);
        load_block(0, blk(i + 2));
        block(1, k0 + 32 * (i + 1));
        load_block(1, blk(i + 3));
    }
    if (i < nblk) block(0, k0 + 32 * i);
    if (i + 1 < nblk) block(1, k0 + 32 * (i + 1));

    // partial (o, m, l) of this split for each head of the group
    if (j < qpg) {
        float *pr = p.part + (((int64_t)b * p.n_q + kvh * qpg + j) * S + split) * (D + 2);
#pragma unroll
        for (int t = 0; t < NT; ++t) *(f32x4 *)(pr + 16 * t + 4 * g) = o[t];
        if (g == 0) {
            pr[D] = m_run;
            pr[D + 1] = l_run;
        }
    }
}

// merge: one workgroup of D threads per (sequence, query head); thread t
// owns dimension t.  Weights exp2(m_s - M) and L = sum_s w_s l_s, then the
// weighted sum of the split outputs in split order; every split's value is
// requested before any is used.
template <int D>
__global__ __launch_bounds__(D) void k_attn_merge(AttnDecodeParams p) {
    constexpr int SMAX = 64;
    __shared__ float s_w[SMAX];
    __shared__ float s_inv;
    const int t = threadIdx.x;
    const int S = p.splits;
    const int bh = blockIdx.x;                        // b * n_q + head
    const float *ph = p.part + (int64_t)bh * S * (D + 2);
    float ov[SMAX];
#pragma unroll
    for (int sp = 0; sp < SMAX; ++sp) ov[sp] = ph[(sp < S ? sp : 0) * (D + 2) + t];
    if (t < 64) {
        const float msr = ph[(t < S ? t : 0) * (D + 2) + D], lsr = ph[(t < S ? t : 0) * (D + 2) + D + 1];
        const float ms = t < S ? msr : -INFINITY;
        const float ls = t < S ? lsr : 0.f;
        const float M = wave_max(ms);
        const float w = ms == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(ms - M);
        const float L = wave_sum(w * ls);
        s_w[t] = w;
        if (t == 0) s_inv = 1.0f / L;
    }
    __syncthreads();
    float acc = 0.f;
#pragma unroll
    for (int sp = 0; sp < SMAX; ++sp) acc += sp < S ? s_w[sp] * ov[sp] : 0.f;
    p.out[(int64_t)bh * D + t] = acc * s_inv;
}

void launch_attn_decode(const AttnDecodeParams &p, hipStream_t s) {
    const int grid = p.B * p.n_kv * p.splits;
    if (p.d == 128) {
        hipLaunchKernelGGL(k_attn_decode<128>, dim3(grid), dim3(64), 0, s, p);
        hipLaunchKernelGGL(k_attn_merge<128>, dim3(p.B * p.n_q), dim3(128), 0, s, p);
    } else {
        hipLaunchKernelGGL(k_attn_decode<64>, dim3(grid), dim3(64), 0, s, p);
        hipLaunchKernelGGL(k_attn_merge<64>, dim3(p.B * p.n_q), dim3(64), 0, s, p);
    }
}

}  // namespace pipo
