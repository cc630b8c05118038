// Grouped-query flash-decode over the latent KV cache (one query position per
// sequence), split along the key axis.
//
// One wave per (sequence, KV group, split).  The group's query heads are the
// 16 columns of the MFMA tiles (unused columns are zero): scores are computed
// transposed, S^T[key][head] = K Q^T, 16 keys per tile, so each lane's
// accumulator holds one head; online softmax runs per column; the
// probabilities, held as (4g + v, 16 + 4g + v) for lane group g, are already
// the B operand of O^T[dim][head] += V^T P^T because the V cache stores each
// 32-key tile in that key order (vslot in device_common.h).  The query and
// the probabilities enter the MFMAs as bf16 pairs hi + lo (two MFMAs each),
// so only the bf16 KV cache itself limits the precision.  Per-split results
// (m, l, o) are merged in split order in one of three ways: when the
// (sequence, KV group) pairs fill the machine they stay in one workgroup
// whose waves are the splits and merge through LDS; up to 24 splits the
// splits of a pair run on one XCD and the last to finish merges their
// records through that XCD's L2; otherwise a second kernel merges the
// records per head (the kernel boundary makes every split's record visible).
#include "device_common.h"
#include <vector>

#include "kernels.h"

namespace pipo {

// The merge of one (sequence, KV group) by one wave: the records of its qpg
// heads and S splits ([qpg][S] in the partial buffer).  16 lanes take a head,
// D / 16 dimensions each, four heads at a time; the splits go in split order,
// XU at a time, with the running maximum M and the sums L and o rescaled by
// exp2(M_old - M_new) as it rises; then o / L.
template <int D>
__device__ void xl_merge(const AttnDecodeParams &p, int b, int kvh, int qpg, int S, int lane) {
    constexpr int RS = attn_part_stride(D), DPL = D / 16, XU = 12;
    const float *rec = p.part + ((int64_t)b * p.n_q + kvh * qpg) * S * RS;   // [qpg][S][RS]
    const int d0 = (lane & 15) * DPL;
    for (int h0 = 0; h0 < qpg; h0 += 4) {
        const int hj = h0 + (lane >> 4);
        const float *rh = rec + (int64_t)(hj < qpg ? hj : 0) * S * RS;
        float M = -INFINITY, L = 0.f, acc[DPL];
#pragma unroll
        for (int k = 0; k < DPL; ++k) acc[k] = 0.f;
        for (int s0 = 0; s0 < S; s0 += XU) {
            float2 ml[XU];
            float4 ov[XU][DPL / 4];
#pragma unroll
            for (int u = 0; u < XU; ++u) {
                const float *r = rh + (int64_t)min(s0 + u, S - 1) * RS;
                ml[u] = *(const float2 *)(r + D);
#pragma unroll
                for (int k = 0; k < DPL / 4; ++k) ov[u][k] = ((const float4 *)(r + d0))[k];
            }
            float Mn = M;
#pragma unroll
            for (int u = 0; u < XU; ++u) Mn = fmaxf(Mn, s0 + u < S ? ml[u].x : -INFINITY);
            const float sc = Mn == -INFINITY ? 1.f : __builtin_amdgcn_exp2f(M - Mn);
            L *= sc;
#pragma unroll
            for (int k = 0; k < DPL; ++k) acc[k] *= sc;
#pragma unroll
            for (int u = 0; u < XU; ++u) {
                const float w = (s0 + u < S && ml[u].x != -INFINITY) ? __builtin_amdgcn_exp2f(ml[u].x - Mn) : 0.f;
                L += w * ml[u].y;
#pragma unroll
                for (int k = 0; k < DPL / 4; ++k) {
                    acc[4 * k + 0] += w * ov[u][k].x;
                    acc[4 * k + 1] += w * ov[u][k].y;
                    acc[4 * k + 2] += w * ov[u][k].z;
                    acc[4 * k + 3] += w * ov[u][k].w;
                }
            }
            M = Mn;
        }
        if (hj < qpg) {
            const float inv = 1.0f / L;
            float *o = p.out + ((int64_t)b * p.n_q + kvh * qpg + hj) * D + d0;
#pragma unroll
            for (int k = 0; k < DPL / 4; ++k)
                *(float4 *)(o + 4 * k) = make_float4(acc[4 * k] * inv, acc[4 * k + 1] * inv, acc[4 * k + 2] * inv,
                                                     acc[4 * k + 3] * inv);
        }
    }
}

// FUSED: the QKV GEMV left its k-range partial sums [R][B][nqkv] (rows in its
// strip order: strip t of a q or k head holds dims 8t..8t+7, then their RoPE
// partners d/2+8t..; v heads in order).  Every split adds the ranges of its
// group's query rows in range order and applies RoPE (staging the rotated
// rows in LDS); the split that holds the new position also adds that
// position's key and value rows and rotates the key, scores the new key from
// registers (one online-softmax step after its blocks, which stop before it)
// and stores the key and value to the cache at its end, for later steps.
// NW: waves per workgroup.  1: one wave per (sequence, KV group, split),
// partial records to global memory, merged on the XCD (xl_ctr) or by
// k_attn_merge.  NW > 1: one workgroup per (sequence, KV group) whose NW
// waves are its splits; their partials are combined in LDS in split order and
// the workgroup writes the output rows.  At most 256 registers a lane, so
// that two waves fit on a SIMD (9B at batch 8: 2.86 ms of attention per pair
// step this way, 2.88 with the 278 the compiler chooses otherwise).
template <int D, bool FUSED, int NW>
__global__ __launch_bounds__(64 * NW, 2) void k_attn_decode(AttnDecodeParams p) {
    constexpr int NC = D / 32;   // 32-wide d chunks (QK^T k-steps)
    constexpr int NT = D / 16;   // 16-wide d tiles (PV output tiles)
    const int lane = threadIdx.x & 63, j = lane & 15, g = lane >> 4;
    const int wave = NW > 1 ? (int)threadIdx.x >> 6 : 0;
    const int S = NW > 1 ? NW : p.splits;
    constexpr int RS = attn_part_stride(D);
    // XCD-local merge: workgroup i runs on XCD i mod 8, so pair (sequence, KV
    // group) k takes workgroups ((k / 8) S + split) 8 + k mod 8
    const bool xl = NW == 1 && p.xl_ctr != nullptr;
    const int xm = (int)blockIdx.x >> 3;
    const int split = NW > 1 ? wave : xl ? xm % S : (int)blockIdx.x % S;
    const int bk = NW > 1 ? (int)blockIdx.x : xl ? (xm / S) * 8 + ((int)blockIdx.x & 7) : (int)blockIdx.x / S;
    if (xl && bk >= p.B * p.n_kv) return;   // (a one-wave workgroup: no barrier to leave)
    const int b = bk / p.n_kv, kvh = bk - b * p.n_kv;
    const int qpg = p.n_q / p.n_kv;
    // splits own whole 32-key blocks: split s takes blocks [s*nb/S, (s+1)*nb/S)
    const int len = p.pos[b] + 1;
    const int nb = (len + 31) >> 5;
    const int k0 = ((split * nb) / S) * 32;
    // FUSED: the last split takes the new key (position len - 1) from
    // registers, after its blocks, so its blocks stop before it
    const int k1 = min(len - ((FUSED && split == S - 1) ? 1 : 0), (((split + 1) * nb) / S) * 32);
    const float scale = 1.4426950408889634f / sqrtf((float)D);

    const uint16_t *kbase = p.kc + (int64_t)b * p.kv_bstride + (int64_t)kvh * p.lmax_pad * D;
    const uint16_t *vbase = p.vc + (int64_t)b * p.kv_bstride + (int64_t)kvh * p.lmax_pad * D;
    constexpr int HS = D / 16;                    // strips per head in the QKV row order
    const int jq = j < qpg ? j : 0;               // unused columns take head 0 (zeroed below)
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

    float4 qr[NC][2];
    __shared__ float s_new_all[NW][2][D];   // FUSED, last split: the new key and value (bf16 values)
    float (&s_new)[2][D] = s_new_all[wave];
    float s_key = 0.f;                 // FUSED, last split: the new key's scaled score
    if constexpr (FUSED) {
        // LDS: the group's rotated query rows [qpg][D] (qpg * D <= 1024) and,
        // for the last split, the new key and value (bf16 values)
        __shared__ float s_q_all[NW][1024];
        float (&s_q)[1024] = s_q_all[wave];
        const bool hold = split == S - 1;
        const int R = p.ksplit, pos = len - 1;
        const int64_t NB = (int64_t)p.B * p.nqkv;
        const float *P = p.qkv_part + (int64_t)b * p.nqkv;
        const int qs = p.n_q * HS, kvs = p.n_kv * HS;
        // The group's query rows are contiguous (qpg heads of D rows each).
        // A strip's rows 4 qq .. 4 qq + 3 (dims 8 t + 4 qq ..) pair with rows
        // 8 + 4 qq .. (their RoPE partners): lane l takes quarter-pairs l and
        // l + 64, so its RoPE needs only its own loads.
        const int npair = qpg * D / 8;
        const float *Pq = P + (int64_t)kvh * qpg * D;
        int qrow[2];
#pragma unroll
        for (int pp = 0; pp < 2; ++pp) {
            const int pi = min(lane + 64 * pp, npair - 1);
            qrow[pp] = (pi >> 1) * 16 + 4 * (pi & 1);
        }
        // new key and value (last split, lane l < D/2: dims l and l + D/2)
        const bool kvl = hold && lane < D / 2;
        const int jd = lane & (D / 2 - 1);
        const int krow = (qs + kvh * HS + (jd >> 3)) * 16 + (jd & 7);
        const int vrow = (qs + kvs + kvh * HS) * 16 + jd;
        // the partial sums, added in range order
        static_assert(kAttnFusedRanges == 4, "one round trip of four ranges");
        float4 qa[2][2], u[4][2][2];
        float ka = 0.f, kb = 0.f, va = 0.f, vb = 0.f, w[4][4];
        auto load_parts = [&](int r0) {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int64_t off = (int64_t)min(r0 + e, R - 1) * NB;
#pragma unroll
                for (int pp = 0; pp < 2; ++pp) {
                    u[e][pp][0] = *(const float4 *)(Pq + off + qrow[pp]);
                    u[e][pp][1] = *(const float4 *)(Pq + off + qrow[pp] + 8);
                }
                // (every lane: a branch here would wait for them one range at a time)
                w[e][0] = P[off + krow];
                w[e][1] = P[off + krow + 8];
                w[e][2] = P[off + vrow];
                w[e][3] = P[off + vrow + D / 2];
            }
        };
        // ranges past R add zero (selects, not branches, so that no load is
        // moved into a branch)
        auto add_parts = [&](int r0) {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const bool on = r0 + e < R;
#pragma unroll
                for (int pp = 0; pp < 2; ++pp)
#pragma unroll
                    for (int h = 0; h < 2; ++h) {
                        qa[pp][h].x += on ? u[e][pp][h].x : 0.f; qa[pp][h].y += on ? u[e][pp][h].y : 0.f;
                        qa[pp][h].z += on ? u[e][pp][h].z : 0.f; qa[pp][h].w += on ? u[e][pp][h].w : 0.f;
                    }
                ka += on ? w[e][0] : 0.f;
                kb += on ? w[e][1] : 0.f;
                va += on ? w[e][2] : 0.f;
                vb += on ? w[e][3] : 0.f;
            }
        };
        // the ranges (at most kAttnFusedRanges) and the RoPE values go out
        // before the first blocks' loads, so that waiting for them leaves the
        // blocks in flight
        load_parts(0);
        float4 cq[2], sq[2];
#pragma unroll
        for (int pp = 0; pp < 2; ++pp) {
            const int pi = min(lane + 64 * pp, npair - 1);
            const int jr = ((pi >> 1) % HS) * 8 + 4 * (pi & 1);
            cq[pp] = *(const float4 *)(p.rope_cos + (int64_t)pos * (D / 2) + jr);
            sq[pp] = *(const float4 *)(p.rope_sin + (int64_t)pos * (D / 2) + jr);
        }
        const float ck = p.rope_cos[(int64_t)pos * (D / 2) + jd], sk = p.rope_sin[(int64_t)pos * (D / 2) + jd];
        __builtin_amdgcn_sched_barrier(0);
        load_block(0, blk(0));
        load_block(1, blk(1));
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int pp = 0; pp < 2; ++pp) qa[pp][0] = qa[pp][1] = make_float4(0.f, 0.f, 0.f, 0.f);
        add_parts(0);
        // RoPE (dim i < D/2 pairs with i + D/2 at frequency index i) into the
        // natural [head][dim] order
#pragma unroll
        for (int pp = 0; pp < 2; ++pp) {
            const int pi = lane + 64 * pp;
            if (pi < npair) {
                const int hl = (pi >> 1) / HS, jr = ((pi >> 1) % HS) * 8 + 4 * (pi & 1);
                const float4 a = qa[pp][0], o = qa[pp][1], cs = cq[pp], sn = sq[pp];
                *(float4 *)&s_q[hl * D + jr] = make_float4(a.x * cs.x - o.x * sn.x, a.y * cs.y - o.y * sn.y,
                                                          a.z * cs.z - o.z * sn.z, a.w * cs.w - o.w * sn.w);
                *(float4 *)&s_q[hl * D + D / 2 + jr] = make_float4(o.x * cs.x + a.x * sn.x, o.y * cs.y + a.y * sn.y,
                                                                  o.z * cs.z + a.z * sn.z, o.w * cs.w + a.w * sn.w);
            }
        }
        if (kvl) {
            // the new key, rotated and rounded to bf16 as the cache holds it
            s_new[0][jd] = __uint_as_float(f2bf(ka * ck - kb * sk) << 16);
            s_new[0][jd + D / 2] = __uint_as_float(f2bf(kb * ck + ka * sk) << 16);
            s_new[1][jd] = __uint_as_float(f2bf(va) << 16);
            s_new[1][jd + D / 2] = __uint_as_float(f2bf(vb) << 16);
        }
        __syncthreads();
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            qr[c][0] = *(const float4 *)&s_q[jq * D + 32 * c + 8 * g];
            qr[c][1] = *(const float4 *)&s_q[jq * D + 32 * c + 8 * g + 4];
        }
        if (hold) {
            // the new key's score per head, from the fp32 query
            float dot = 0.f;
#pragma unroll
            for (int c = 0; c < NC; ++c)
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    const float *kn = &s_new[0][32 * c + 8 * g + 4 * h];
                    dot += qr[c][h].x * kn[0] + qr[c][h].y * kn[1] + qr[c][h].z * kn[2] + qr[c][h].w * kn[3];
                }
            dot += __shfl_xor(dot, 16);
            dot += __shfl_xor(dot, 32);
            s_key = dot * scale;
        }
    } else {
        // the query rows and the first two blocks are requested together,
        // before any of them is waited for
        const float4 *qp = (const float4 *)(p.q + ((int64_t)b * p.n_q + kvh * qpg + jq) * D + 8 * g);
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            qr[c][0] = qp[8 * c];
            qr[c][1] = qp[8 * c + 1];
        }
        load_block(0, blk(0));
        load_block(1, blk(1));
    }
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

    if (FUSED && split == S - 1) {
        // the new key (its score taken before the blocks): one online-softmax
        // step and its value row
        const float sv = s_key;
        const float m_new = fmaxf(m_run, sv);
        const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
        const float pe = __builtin_amdgcn_exp2f(sv - m_new);
        l_run = l_run * alpha + pe;
        m_run = m_new;
#pragma unroll
        for (int t = 0; t < NT; ++t)
#pragma unroll
            for (int v = 0; v < 4; ++v) o[t][v] = o[t][v] * alpha + pe * s_new[1][16 * t + 4 * g + v];
        // the new key and value into the cache for later steps (stored only
        // now: a store pending among the block loads would make the compiler
        // wait for every load in flight)
        if (lane < D / 2) {
            const int pos = len - 1;
            uint16_t *kw = (uint16_t *)kbase, *vw = (uint16_t *)vbase;
            kw[tiled_index(pos, lane, D)] = (uint16_t)(__float_as_uint(s_new[0][lane]) >> 16);
            kw[tiled_index(pos, lane + D / 2, D)] = (uint16_t)(__float_as_uint(s_new[0][lane + D / 2]) >> 16);
            vw[((int64_t)(pos >> 5) * D + lane) * 32 + vslot(pos & 31)] = (uint16_t)(__float_as_uint(s_new[1][lane]) >> 16);
            vw[((int64_t)(pos >> 5) * D + lane + D / 2) * 32 + vslot(pos & 31)] =
                (uint16_t)(__float_as_uint(s_new[1][lane + D / 2]) >> 16);
        }
    }
    if constexpr (NW == 1) {
        // partial (o, m, l) of this split for each head of the group
        if (j < qpg) {
            float *pr = p.part + (((int64_t)b * p.n_q + kvh * qpg + j) * S + split) * RS;
#pragma unroll
            for (int t = 0; t < NT; ++t) *(f32x4 *)(pr + 16 * t + 4 * g) = o[t];
            if (g == 0) {
                pr[D] = m_run;
                pr[D + 1] = l_run;
            }
        }
        if (xl) {
            // the last split of this pair to finish merges it: its stores are
            // acknowledged by L2 before it counts itself in (the pair's other
            // splits wrote theirs to the same L2; every record is whole cache
            // lines, and no load of them happened on this CU before, so the
            // loads below see them)
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
            int old = 0;
            if (lane == 0) old = __hip_atomic_fetch_add(p.xl_ctr + bk, 1, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_WORKGROUP);
            old = __builtin_amdgcn_readfirstlane(old);
            if (old == S - 1) {
                if (lane == 0) __hip_atomic_store(p.xl_ctr + bk, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
                xl_merge<D>(p, b, kvh, qpg, S, lane);
            }
        }
    } else {
        // the splits' (o, m, l) through LDS, merged as k_attn_merge does:
        // weights exp2(m_s - M), L = sum_s w_s l_s, the weighted outputs
        // added in split order
        __shared__ float red[NW][16][D + 2];
        if (j < qpg) {
#pragma unroll
            for (int t = 0; t < NT; ++t)
#pragma unroll
                for (int v = 0; v < 4; ++v) red[wave][j][16 * t + 4 * g + v] = o[t][v];
            if (g == 0) {
                red[wave][j][D] = m_run;
                red[wave][j][D + 1] = l_run;
            }
        }
        __syncthreads();
        for (int e = threadIdx.x; e < qpg * D; e += 64 * NW) {
            const int hj = e / D, dim = e - hj * D;
            float M = -INFINITY;
#pragma unroll
            for (int w = 0; w < NW; ++w) M = fmaxf(M, red[w][hj][D]);
            float L = 0.f, acc = 0.f;
#pragma unroll
            for (int w = 0; w < NW; ++w) {
                const float mw = red[w][hj][D];
                const float ww = mw == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(mw - M);
                L += ww * red[w][hj][D + 1];
                acc += ww * red[w][hj][dim];
            }
            p.out[((int64_t)b * p.n_q + kvh * qpg + hj) * D + dim] = acc * (1.0f / L);
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
    constexpr int RS = attn_part_stride(D);
    const float *ph = p.part + (int64_t)bh * S * RS;
    float ov[SMAX];
#pragma unroll
    for (int sp = 0; sp < SMAX; ++sp) ov[sp] = ph[(sp < S ? sp : 0) * RS + t];
    if (t < 64) {
        const float msr = ph[(t < S ? t : 0) * RS + D], lsr = ph[(t < S ? t : 0) * RS + D + 1];
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

__global__ __launch_bounds__(64) void k_xcd_probe(int *out) {
    if (threadIdx.x == 0) {
        unsigned x;
        asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(x));
        out[blockIdx.x] = (int)(x & 0xF);
    }
}

hipError_t probe_xcd_round_robin(hipStream_t s, bool *ok) {
    constexpr int n = 2048;
    *ok = false;
    int *d = nullptr;
    hipError_t e = hipMalloc(&d, n * sizeof(int));
    if (e != hipSuccess) return e;
    std::vector<int> h(n);
    hipLaunchKernelGGL(k_xcd_probe, dim3(n), dim3(64), 0, s, d);
    e = hipGetLastError();
    if (e == hipSuccess) e = hipMemcpyAsync(h.data(), d, n * sizeof(int), hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    hipFree(d);
    if (e != hipSuccess) return e;
    bool good = true, seen[16] = {};
    for (int i = 0; i < 8; ++i) {
        good = good && !seen[h[i]];
        seen[h[i]] = true;
    }
    for (int i = 8; i < n; ++i) good = good && h[i] == h[i % 8];
    *ok = good;
    return hipSuccess;
}

void launch_attn_decode(const AttnDecodeParams &p, hipStream_t s) {
    const bool fused = p.qkv_part != nullptr;
    if (p.splits == kAttnWgSplits) {   // one workgroup per (sequence, KV group), no merge launch
        const int grid = p.B * p.n_kv;
        constexpr int NW = kAttnWgSplits;
        if (p.d == 128) {
            if (fused) hipLaunchKernelGGL((k_attn_decode<128, true, NW>), dim3(grid), dim3(64 * NW), 0, s, p);
            else hipLaunchKernelGGL((k_attn_decode<128, false, NW>), dim3(grid), dim3(64 * NW), 0, s, p);
        } else {
            if (fused) hipLaunchKernelGGL((k_attn_decode<64, true, NW>), dim3(grid), dim3(64 * NW), 0, s, p);
            else hipLaunchKernelGGL((k_attn_decode<64, false, NW>), dim3(grid), dim3(64 * NW), 0, s, p);
        }
        return;
    }
    const bool xl = p.xl_ctr != nullptr;
    const int pairs = p.B * p.n_kv;
    const int grid = xl ? 8 * p.splits * ((pairs + 7) / 8) : pairs * p.splits;
    if (p.d == 128) {
        if (fused) hipLaunchKernelGGL((k_attn_decode<128, true, 1>), dim3(grid), dim3(64), 0, s, p);
        else hipLaunchKernelGGL((k_attn_decode<128, false, 1>), dim3(grid), dim3(64), 0, s, p);
        if (!xl) hipLaunchKernelGGL(k_attn_merge<128>, dim3(p.B * p.n_q), dim3(128), 0, s, p);
    } else {
        if (fused) hipLaunchKernelGGL((k_attn_decode<64, true, 1>), dim3(grid), dim3(64), 0, s, p);
        else hipLaunchKernelGGL((k_attn_decode<64, false, 1>), dim3(grid), dim3(64), 0, s, p);
        if (!xl) hipLaunchKernelGGL(k_attn_merge<64>, dim3(p.B * p.n_q), dim3(64), 0, s, p);
    }
}

}  // namespace pipo
