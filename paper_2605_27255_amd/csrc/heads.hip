// Output side of a pair step: the confidence gate and next-pair builder
// (eq. 6 and the PAD fallback of Sec. 3.2), and token selection: temperature
// + top-p, and the evaluation sampler of Sec. 4 (repetition penalty,
// temperature, top-k, top-p).
#include "device_common.h"
#include "kernels.h"

namespace pipo {

// Set token t's bit in a penalised-token bitmap row (ids outside [0, V) are
// not tokens and are skipped).
__device__ __forceinline__ void seen_set(uint32_t *row, int32_t t, int V) {
    if (t >= 0 && t < V) atomicOr(row + (t >> 5), 1u << (t & 31));
}

__global__ __launch_bounds__(256) void k_seen_mark(const int32_t *tokens, int n, const int32_t *ntok, int V,
                                                   uint32_t *seen, int seen_words) {
    const int b = blockIdx.y;
    const int i = blockIdx.x * 256 + threadIdx.x;
    if (i < (ntok ? ntok[b] : n)) seen_set(seen + (int64_t)b * seen_words, tokens[(int64_t)b * n + i], V);
}

void launch_seen_mark(const int32_t *tokens, int n, const int32_t *ntok, int B, int V, uint32_t *seen, int seen_words,
                      hipStream_t s) {
    hipLaunchKernelGGL(k_seen_mark, dim3((n + 255) / 256, B), dim3(256), 0, s, tokens, n, ntok, V, seen, seen_words);
}

struct PairOut { int32_t tok_b, tok_d; float conf; int32_t accept; };

// One workgroup per sequence: s = w_c . RMSNorm([h_b; h_d]) * g_c,
// c = sigmoid(s), accept iff c >= tau; next pair = (b, accept ? d : PAD).
__global__ __launch_bounds__(512) void k_gate(GateParams p) {
    __shared__ float red[8];
    __shared__ float s_sc;
    const int b = blockIdx.x, lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int H = p.H;
    const bool mlp = p.conf_h != nullptr;   // App. B.3: w2 . SiLU(W1 RMSNorm([h_b; h_d])), hidden precomputed
    if (wave == 0) {
        float a = 0.f;
        for (int i = lane; i < p.nss_b; i += 64) a += p.ss_b[b * p.nss_b + i];
        for (int i = lane; i < p.nss_d; i += 64) a += p.ss_d[b * p.nss_d + i];
        a = wave_sum(a);
        if (lane == 0) s_sc = mlp ? 1.0f : rsqrtf(a / (float)(2 * H) + p.eps);
    }
    float dot = 0.f;
    if (mlp) {
#pragma unroll 4
        for (int k = threadIdx.x; k < H; k += 512) dot += p.conf_w2[k] * p.conf_h[(int64_t)b * H + k];
    } else {
#pragma unroll 4
        for (int k = threadIdx.x; k < 2 * H; k += 512) {
            const float u = k < H ? p.hb[(int64_t)b * H + k] : p.hd[(int64_t)b * H + k - H];
            dot += p.w_conf[k] * p.g_conf[k] * u;
        }
    }
    dot = wave_sum(dot);
    if (lane == 0) red[wave] = dot;
    __syncthreads();
    if (threadIdx.x == 0) {
        const float s = (((red[0] + red[1]) + (red[2] + red[3])) + ((red[4] + red[5]) + (red[6] + red[7]))) * s_sc;
        const float c = 1.0f / (1.0f + expf(-s));
        const int acc = c >= p.tau ? 1 : 0;
        const int32_t tb = argmax_key_id(p.best_b[b]);
        const int32_t td = argmax_key_id(p.best_d[b]);
        if (p.seen) {   // the tokens this step took as input were emitted: later steps penalise them
            uint32_t *row = p.seen + (int64_t)b * p.seen_words;
            seen_set(row, p.pairs[2 * b], p.V);
            if (p.pairs[2 * b + 1] != p.pad_id) seen_set(row, p.pairs[2 * b + 1], p.V);
        }
        PairOut *o = (PairOut *)p.out + b;
        o->tok_b = tb;
        o->tok_d = td;
        o->conf = c;
        o->accept = acc;
        p.pairs[2 * b] = tb;
        p.pairs[2 * b + 1] = acc ? td : p.pad_id;
        if (p.advance) p.pos[b] += 1;
        p.step[b] += 1;
        p.best_b[b] = 0;
        p.best_d[b] = 0;
    }
}

void launch_gate(const GateParams &p, hipStream_t s) {
    hipLaunchKernelGGL(k_gate, dim3(p.B), dim3(512), 0, s, p);
}

// ---------------------------------------------------------------------------
// Embedding rows of the step's input tokens: x[b] = E[first token] (regular
// decoding, the paper's baseline of Sec. 4.3), or E[a] + E[b] of the pending
// pair (`both`: the skip path of the MLP compressor), in fp32 with the
// sum-of-squares part of every 16-element strip, as the RMSNorm prologue of
// the decode GEMM reads them.
__global__ __launch_bounds__(256) void k_embed_step(const int32_t *pairs, const uint16_t *embed, int H, int V,
                                                    float *x, float *ss, int both) {
    const int b = blockIdx.x;
    const int row = clamp_id(pairs[2 * b], V);
    const int row2 = clamp_id(pairs[2 * b + 1], V);
    for (int c = threadIdx.x; c < (H >> 3); c += 256) {
        const int k = c << 3;
        const u32x4 v = *(const u32x4 *)(embed + tiled_index(row, k, H));
        float f[8] = {bf_lo(v[0]), bf_hi(v[0]), bf_lo(v[1]), bf_hi(v[1]),
                      bf_lo(v[2]), bf_hi(v[2]), bf_lo(v[3]), bf_hi(v[3])};
        if (both) {
            const u32x4 w = *(const u32x4 *)(embed + tiled_index(row2, k, H));
            f[0] += bf_lo(w[0]); f[1] += bf_hi(w[0]); f[2] += bf_lo(w[1]); f[3] += bf_hi(w[1]);
            f[4] += bf_lo(w[2]); f[5] += bf_hi(w[2]); f[6] += bf_lo(w[3]); f[7] += bf_hi(w[3]);
        }
        float4 *dst = (float4 *)(x + (int64_t)b * H + k);
        dst[0] = make_float4(f[0], f[1], f[2], f[3]);
        dst[1] = make_float4(f[4], f[5], f[6], f[7]);
        float q = 0.f;
#pragma unroll
        for (int i = 0; i < 8; ++i) q += f[i] * f[i];
        q += __shfl_xor(q, 1);          // the strip's other half (chunk c ^ 1)
        if ((c & 1) == 0) ss[(int64_t)b * (H >> 4) + (c >> 1)] = q;
    }
}

void launch_embed_step(const int32_t *pairs, const uint16_t *embed, int H, int V, float *x, float *ss, int B,
                       int both, hipStream_t s) {
    hipLaunchKernelGGL(k_embed_step, dim3(B), dim3(256), 0, s, pairs, embed, H, V, x, ss, both);
}

// Step output: the selected token, which is also the next step's input.
// With a bitmap, the step's input token joins the sequence's penalised set.
__global__ void k_regular_out(uint64_t *best, int32_t *out_tok, int32_t *pairs, int32_t pad_id, int32_t *pos,
                              int32_t *step, int advance, int B, uint32_t *seen, int seen_words, int V) {
    const int b = blockIdx.x * blockDim.x + threadIdx.x;
    if (b >= B) return;
    if (seen) seen_set(seen + (int64_t)b * seen_words, pairs[2 * b], V);
    const int32_t t = argmax_key_id(best[b]);
    out_tok[b] = t;
    pairs[2 * b] = t;
    pairs[2 * b + 1] = pad_id;
    if (advance) pos[b] += 1;
    step[b] += 1;
    best[b] = 0;
}

void launch_regular_out(uint64_t *best, int32_t *out_tok, int32_t *pairs, int32_t pad_id, int32_t *pos,
                        int32_t *step, int advance, int B, uint32_t *seen, int seen_words, int V, hipStream_t s) {
    hipLaunchKernelGGL(k_regular_out, dim3((B + 63) / 64), dim3(64), 0, s, best, out_tok, pairs, pad_id, pos, step,
                       advance, B, seen, seen_words, V);
}

// ---------------------------------------------------------------------------
// Temperature + top-p selection, one 1024-thread workgroup per sequence.
//   e_j = exp((l_j - max l) / T) (the hardware exp2; values below the normal
//   range flush to zero, as their fixed-point masses round to zero anyway);
//   masses are fixed point, E_j = round(e_j 2^40),
//   so every sum is an exact integer sum (order independent).
//   theta* = the largest e-value whose upper mass sum_{e_i >= theta} E_i
//   reaches top_p * sum E: found exactly by a 4-pass radix select over the
//   float bit patterns of e (positive floats order like their bits).
//   nucleus N = {j : e_j >= theta*}, mass M; t = floor(u M); the token is the
//   first id, scanning upwards through N, whose running mass exceeds t.
// The evaluation sampler (EVAL) first replaces every penalised logit l by
// l / theta_r if l > 0, else l theta_r (theta_r = rep_penalty), and with
// top_k keeps the tokens whose penalised logit is at least the k-th largest
// (ties kept): a 4-pass radix select for the k-th largest over an order-
// preserving integer image of the floats; top-p then runs on the kept set.
// ---------------------------------------------------------------------------
constexpr int kSampThreads = 1024;

__device__ __forceinline__ uint64_t shfl_up_u64(uint64_t v, int d) {
    uint32_t lo = __shfl_up((uint32_t)v, d), hi = __shfl_up((uint32_t)(v >> 32), d);
    return ((uint64_t)hi << 32) | lo;
}

// round(e 2^40) for e in [0, 1]: exact in double, rounded to nearest even,
// converted without branches (so the loads of a pass stay in flight)
__device__ __forceinline__ uint64_t fixed_mass(float e) {
    return (uint64_t)__builtin_rint((double)e * 1099511627776.0);   // 2^40
}

// Unsigned image of a float that orders like the float (-0 taken as +0).
__device__ __forceinline__ uint32_t order_key(float f) {
    const uint32_t u = __float_as_uint(f + 0.0f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Wave w of the workgroup owns the contiguous ids [w R, (w + 1) R), R a
// multiple of 256, read as 256-element sub-tiles (lane l: ids base + 4 l ..
// base + 4 l + 3, one float4), so every pass is coalesced and id order is
// (wave, sub-tile, lane, element).
constexpr int kSampWaves = kSampThreads / 64;

template <bool EVAL>
__global__ __launch_bounds__(kSampThreads) void k_sample(SampleParams p) {
    __shared__ unsigned long long hist[kSampWaves][256];
    __shared__ float s_red[kSampWaves];
    __shared__ unsigned long long s_u64[kSampWaves];
    __shared__ uint32_t s_prefix;
    __shared__ unsigned long long s_above, s_mass;
    __shared__ int s_all;

    const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const float *lg = p.logits + (int64_t)b * p.V;
    const int V = p.V;
    const int R = ((V + kSampWaves * 256 - 1) / (kSampWaves * 256)) * 256;   // ids per wave
    const int w0 = wave * R;
    // penalised ids besides the bitmap: the step's input pair (the second
    // unless PAD) and the extra token; -1: none
    int ex0 = -1, ex1 = -1, ex2 = -1;
    const uint32_t *seen = nullptr;
    if constexpr (EVAL) {
        if (p.seen) seen = p.seen + (int64_t)b * p.seen_words;
        if (p.pairs) {
            ex0 = p.pairs[2 * b];
            ex1 = p.pairs[2 * b + 1] == p.pad_id ? -1 : p.pairs[2 * b + 1];
        }
        if (p.extra_key) ex2 = argmax_key_id(p.extra_key[b]);
    }
    // The four logits of this lane in sub-tile t (ids past V read id 0,
    // masked).  EVAL: the first pass reads the raw logits, applies the
    // penalty and keeps the penalised row in p.pen (each lane rereads only
    // what it wrote itself); every later pass reads that row.
    const float *src = lg;
    float *pen = EVAL ? p.pen + (int64_t)b * V : nullptr;
    auto load4 = [&](int t, float (&v)[4]) {
        const int id = w0 + t * 256 + 4 * lane;
        const float4 q = *(const float4 *)(src + (id + 3 < V ? id : 0));
        v[0] = q.x; v[1] = q.y; v[2] = q.z; v[3] = q.w;
    };
    auto penalise = [&](int t, float (&v)[4]) {
        const int id = w0 + t * 256 + 4 * lane;
        const uint32_t bits = (seen && id < V) ? seen[id >> 5] >> (id & 31) : 0u;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int j = id + e;
            if (((bits >> e) & 1u) || j == ex0 || j == ex1 || j == ex2)
                v[e] = v[e] > 0.f ? v[e] / p.rep_penalty : v[e] * p.rep_penalty;
        }
        if (id + 3 < V) *(float4 *)(pen + id) = make_float4(v[0], v[1], v[2], v[3]);
    };
    // V is a multiple of 16, so a lane's four ids are all in range or all out.
    // Conditions are combined with & and masses masked arithmetically (no
    // short-circuit, no select around a load's use): otherwise the compiler
    // sinks each load into its branch and a pass keeps one load in flight.
    auto valid = [&](int t, int e) { (void)e; return w0 + t * 256 + 4 * lane < V; };
    auto masked = [](bool ok, uint64_t m) { return m & (0ull - (uint64_t)ok); };
    const int nt = R / 256;
    // every pass: four sub-tiles' loads issued together, then their use
    auto for_tiles = [&](auto &&f) {
        int t = 0;
        for (; t + 4 <= nt; t += 4) {
            float v[4][4];
#pragma unroll
            for (int u = 0; u < 4; ++u) load4(t + u, v[u]);
#pragma unroll
            for (int u = 0; u < 4; ++u) f(t + u, v[u]);
        }
        for (; t < nt; ++t) {
            float v[4];
            load4(t, v);
            f(t, v);
        }
    };
    // Suffix sums S_k = sum_{k' >= k} hist[0][k'] of the merged histogram
    // into s_suf (threads 0..255, a reversed wave scan); then each bin tests
    // its own suffix, so the digit is one parallel step instead of a serial
    // 256-step scan.
    __shared__ unsigned long long s_suf[257], s_wtot[4];
    __shared__ int s_dig;
    auto suffix_sums = [&]() {
        unsigned long long x = 0;
        if (tid < 256) {
            x = hist[0][255 - tid];
            for (int d = 1; d < 64; d <<= 1) {
                const unsigned long long y = shfl_up_u64(x, d);
                if (lane >= d) x += y;
            }
            if (lane == 63) s_wtot[wave] = x;
        }
        if (tid == 0) { s_dig = -1; s_suf[256] = 0; }
        __syncthreads();
        if (tid < 256) {
            for (int w = 0; w < wave; ++w) x += s_wtot[w];
            s_suf[255 - tid] = x;
        }
        __syncthreads();
    };

    float mx = -INFINITY;
    for_tiles([&](int t, const float (&v0)[4]) {
        float v[4] = {v0[0], v0[1], v0[2], v0[3]};
        if constexpr (EVAL) penalise(t, v);
#pragma unroll
        for (int e = 0; e < 4; ++e) mx = fmaxf(mx, valid(t, e) ? v[e] : -INFINITY);
    });
    if constexpr (EVAL) src = pen;
    mx = wave_max(mx);
    if (lane == 0) s_red[wave] = mx;
    __syncthreads();
    mx = s_red[0];
    for (int w = 1; w < kSampWaves; ++w) mx = fmaxf(mx, s_red[w]);
    const float kT = 1.4426950408889634f / p.temperature;

    // top-k: kstar = image of the k-th largest penalised logit; kept = key >= kstar
    uint32_t kstar = 0;
    if constexpr (EVAL) {
        if (p.top_k > 0 && p.top_k < V) {
            __shared__ uint32_t s_kpre, s_krem;
            if (tid == 0) { s_kpre = 0; s_krem = (uint32_t)p.top_k; }
            for (int pass = 0; pass < 4; ++pass) {
                const int shift = 24 - 8 * pass;
                for (int i = tid; i < kSampWaves * 256; i += kSampThreads) (&hist[0][0])[i] = 0;
                __syncthreads();
                const uint32_t prefix = s_kpre;
                for_tiles([&](int t, const float (&v)[4]) {
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const uint32_t key = order_key(v[e]);
                        if (valid(t, e) & ((pass == 0) | ((key >> ((shift + 8) & 31)) == prefix)))
                            atomicAdd(&hist[wave][(key >> shift) & 255u], 1ull);
                    }
                });
                __syncthreads();
                if (tid < 256) {
                    unsigned long long h = 0;
                    for (int w = 0; w < kSampWaves; ++w) h += hist[w][tid];
                    hist[0][tid] = h;
                }
                __syncthreads();
                suffix_sums();
                // the digit holding the rank-krem element: the largest d with S_d >= krem
                const uint32_t krem = s_krem;
                if (tid < 256 && s_suf[tid] >= krem) atomicMax(&s_dig, tid);
                __syncthreads();
                if (tid == 0) {
                    const int d = s_dig < 0 ? 0 : s_dig;
                    s_kpre = (prefix << 8) | (uint32_t)d;
                    s_krem = krem - (uint32_t)s_suf[d + 1];
                }
                __syncthreads();
            }
            kstar = s_kpre;
        }
    }
    // kept: in the vocabulary and, with top-k, at least the k-th largest
    auto kept = [&](int t, int e, float v) { return valid(t, e) & (!EVAL || order_key(v) >= kstar); };

    unsigned long long tot = 0;
    for_tiles([&](int t, const float (&v)[4]) {
#pragma unroll
        for (int e = 0; e < 4; ++e)
            tot += masked(kept(t, e, v[e]), fixed_mass(__builtin_amdgcn_exp2f((v[e] - mx) * kT)));
    });
    for (int o = 32; o > 0; o >>= 1) {
        const uint32_t lo = __shfl_xor((uint32_t)tot, o), hi = __shfl_xor((uint32_t)(tot >> 32), o);
        tot += ((unsigned long long)hi << 32) | lo;
    }
    if (lane == 0) s_u64[wave] = tot;
    __syncthreads();
    tot = 0;
    for (int w = 0; w < kSampWaves; ++w) tot += s_u64[w];
    const double target = (double)p.top_p * (double)tot;

    if (tid == 0) { s_prefix = 0; s_above = 0; s_all = 0; }
    for (int pass = 0; pass < 4; ++pass) {
        const int shift = 24 - 8 * pass;
        for (int i = tid; i < kSampWaves * 256; i += kSampThreads) (&hist[0][0])[i] = 0;
        __syncthreads();
        const uint32_t prefix = s_prefix;
        for_tiles([&](int t, const float (&v)[4]) {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const float ev = __builtin_amdgcn_exp2f((v[e] - mx) * kT);
                const uint32_t key = __float_as_uint(ev);
                if (kept(t, e, v[e]) & ((pass == 0) | ((key >> ((shift + 8) & 31)) == prefix)))
                    atomicAdd(&hist[wave][(key >> shift) & 255u], fixed_mass(ev));
            }
        });
        __syncthreads();
        if (tid < 256) {   // merge the per-wave histograms
            unsigned long long h = 0;
            for (int w = 0; w < kSampWaves; ++w) h += hist[w][tid];
            hist[0][tid] = h;
        }
        __syncthreads();
        suffix_sums();
        // beta: the largest digit whose upper mass (the bins above it and
        // itself) reaches the target
        const unsigned long long above = s_above;
        if (tid < 256 && (double)(above + s_suf[tid]) >= target) atomicMax(&s_dig, tid);
        __syncthreads();
        if (tid == 0) {
            const int beta = s_dig;
            if (beta < 0) {   // no value reaches top_p (rounding): every kept token
                s_all = 1;
            } else {
                s_above = above + s_suf[beta + 1];
                s_prefix = (prefix << 8) | (uint32_t)beta;
                s_mass = above + s_suf[beta];
            }
        }
        __syncthreads();
        if (s_all) break;
    }
    const uint32_t theta = s_all ? 0u : s_prefix;
    const unsigned long long M = s_all ? tot : s_mass;

    // u in [0,1) with 24 bits; t = floor(u * M)
    const uint64_t r24 = splitmix64(rng_key(p.seeds[b], 1ull << 33) + 2ull * (uint64_t)p.step[b] + (uint64_t)p.slot) >> 40;
    const unsigned long long tsel = __umul64hi(r24 << 40, M);

    // nucleus mass of each wave's id range, exclusive prefix over waves
    unsigned long long wm = 0;
    for_tiles([&](int t, const float (&v)[4]) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float ev = __builtin_amdgcn_exp2f((v[e] - mx) * kT);
            wm += masked(kept(t, e, v[e]) & (__float_as_uint(ev) >= theta), fixed_mass(ev));
        }
    });
    for (int o = 32; o > 0; o >>= 1) {
        const uint32_t lo = __shfl_xor((uint32_t)wm, o), hi = __shfl_xor((uint32_t)(wm >> 32), o);
        wm += ((unsigned long long)hi << 32) | lo;
    }
    __syncthreads();
    if (lane == 0) s_u64[wave] = wm;
    __syncthreads();
    unsigned long long run = 0;
    for (int w = 0; w < wave; ++w) run += s_u64[w];
    if (wm == 0 || tsel < run || tsel >= run + wm) return;
    // this wave's range holds the target: walk its sub-tiles in id order
    for (int t = 0; t < nt; ++t) {
        float v[4];
        load4(t, v);
        unsigned long long m4[4], loc = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float ev = __builtin_amdgcn_exp2f((v[e] - mx) * kT);
            m4[e] = masked(kept(t, e, v[e]) & (__float_as_uint(ev) >= theta), fixed_mass(ev));
            loc += m4[e];
        }
        unsigned long long inc = loc;
        for (int d = 1; d < 64; d <<= 1) {
            const unsigned long long o = shfl_up_u64(inc, d);
            if (lane >= d) inc += o;
        }
        const unsigned long long excl = run + inc - loc;
        if (loc > 0 && excl <= tsel && tsel < excl + loc) {
            unsigned long long r = excl;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                r += m4[e];
                if (m4[e] > 0 && r > tsel) {
                    p.best[b] = (1ull << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)(w0 + t * 256 + 4 * lane + e));
                    break;
                }
            }
        }
        run += __shfl(inc, 63);
        if (run > tsel) break;
    }
}

// ---------------------------------------------------------------------------
// Temperature + top-p with each row split over `nseg` workgroups, as six
// short kernels (the same arithmetic and decisions as k_sample, so the same
// token): the row max is the argmax key the LM head left in best[b];
// kernels 0-3 each histogram one byte of the e-values' bits (fixed-point
// masses) over their segment, only among the values whose higher bytes
// match the prefix chosen so far, and store the segment's histogram; the
// kernel after each pass adds the segments' histograms in segment order,
// takes that pass's digit, and its segment-0 workgroup records the state
// (prefix, mass above, nucleus mass, total) for the next kernel; kernel 4
// stores each wave's nucleus mass; kernel 5 draws t = floor(u M) and the
// wave whose id range holds it walks its ids in order.  Integer sums, so
// every order of adding gives the same masses.
constexpr int kSegThreads = 256, kSegWaves = 4;

__device__ __forceinline__ float argmax_key_value(uint64_t key) {
    const uint32_t u = (uint32_t)(key >> 32);
    return __uint_as_float((u & 0x80000000u) ? (u & 0x7FFFFFFFu) : ~u);
}

template <int PASS>
__global__ __launch_bounds__(kSegThreads) void k_sample_seg(SampleParams p) {
    __shared__ unsigned long long hist[kSegWaves][256];
    __shared__ unsigned long long s_suf[257], s_wtot[4];
    __shared__ int s_dig;
    __shared__ SampState s_st;
    const int nseg = p.nseg, B = p.B, V = p.V;
    const int b = blockIdx.x / nseg, seg = blockIdx.x - b * nseg;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int R = p.seg_len, RW = R / kSegWaves;              // ids per segment and per wave (multiples of 256)
    const int w0 = seg * R + wave * RW;
    const int nt = RW / 256;
    const float *lg = p.logits + (int64_t)b * V;
    const float mx = argmax_key_value(p.best[b]);
    const float kT = 1.4426950408889634f / p.temperature;
    unsigned long long *H = p.hist + (int64_t)b * 4 * nseg * 256;      // [pass][segment][256]

    // the state before this kernel's pass: the previous kernel's record and
    // the previous pass's histogram (all segments, in segment order)
    if (PASS == 0) {
        if (tid == 0) s_st = SampState{0u, 0, 0ull, 0ull, 0ull};
        __syncthreads();
        if (seg == 0 && tid == 0) p.state[b] = s_st;
    } else if (PASS == 5) {      // the walk takes the final state as kernel 4 recorded it
        if (tid == 0) s_st = p.state[4 * B + b];
        __syncthreads();
    } else {
        if (tid == 0) s_st = p.state[(PASS - 1) * B + b];
        __syncthreads();
        if (!s_st.all) {
            unsigned long long x = 0;
            if (tid < 256) {
                unsigned long long h = 0;
                for (int sg = 0; sg < nseg; ++sg) h += H[((PASS - 1) * nseg + sg) * 256 + (255 - tid)];
                x = h;
                for (int d = 1; d < 64; d <<= 1) {
                    const unsigned long long y = shfl_up_u64(x, d);
                    if (lane >= d) x += y;
                }
                if (lane == 63) s_wtot[wave] = x;
            }
            if (tid == 0) { s_dig = -1; s_suf[256] = 0; }
            __syncthreads();
            if (tid < 256) {
                for (int w = 0; w < wave; ++w) x += s_wtot[w];
                s_suf[255 - tid] = x;
            }
            __syncthreads();
            // pass 0's histogram holds every token: the total mass
            const unsigned long long tot = PASS == 1 ? s_suf[0] : s_st.total;
            const double target = (double)p.top_p * (double)tot;
            const unsigned long long above = s_st.above;
            if (tid < 256 && (double)(above + s_suf[tid]) >= target) atomicMax(&s_dig, tid);
            __syncthreads();
            if (tid == 0) {
                const int beta = s_dig;
                s_st.total = tot;
                if (beta < 0) {
                    s_st.all = 1;
                } else {
                    s_st.above = above + s_suf[beta + 1];
                    s_st.mass = above + s_suf[beta];
                    s_st.prefix = (s_st.prefix << 8) | (uint32_t)beta;
                }
            }
            __syncthreads();
        }
        if (seg == 0 && tid == 0) p.state[PASS * B + b] = s_st;
    }
    const SampState st = s_st;

    auto load4 = [&](int t, float (&v)[4]) {
        const int id = w0 + t * 256 + 4 * lane;
        const float4 q = *(const float4 *)(lg + (id + 3 < V ? id : 0));
        v[0] = q.x; v[1] = q.y; v[2] = q.z; v[3] = q.w;
    };
    auto valid = [&](int t) { return w0 + t * 256 + 4 * lane < V; };
    auto masked = [](bool ok, uint64_t m) { return m & (0ull - (uint64_t)ok); };
    auto for_tiles = [&](auto &&f) {
        int t = 0;
        for (; t + 4 <= nt; t += 4) {
            float v[4][4];
#pragma unroll
            for (int u = 0; u < 4; ++u) load4(t + u, v[u]);
#pragma unroll
            for (int u = 0; u < 4; ++u) f(t + u, v[u]);
        }
        for (; t < nt; ++t) {
            float v[4];
            load4(t, v);
            f(t, v);
        }
    };

    if constexpr (PASS <= 3) {
        if (st.all) return;
        const int shift = 24 - 8 * PASS;
        for (int i = tid; i < kSegWaves * 256; i += kSegThreads) (&hist[0][0])[i] = 0;
        __syncthreads();
        const uint32_t prefix = st.prefix;
        for_tiles([&](int t, const float (&v)[4]) {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const float ev = __builtin_amdgcn_exp2f((v[e] - mx) * kT);
                const uint32_t key = __float_as_uint(ev);
                // pass 0 takes every value (no shift by 32 of a 32-bit key)
                const bool match = PASS == 0 ? true : ((key >> ((32 - 8 * PASS) & 31)) == prefix);
                if (valid(t) & match) atomicAdd(&hist[wave][(key >> shift) & 255u], fixed_mass(ev));
            }
        });
        __syncthreads();
        if (tid < 256) {
            unsigned long long h = 0;
#pragma unroll
            for (int w = 0; w < kSegWaves; ++w) h += hist[w][tid];
            H[(PASS * nseg + seg) * 256 + tid] = h;
        }
        return;
    }
    const uint32_t theta = st.all ? 0u : st.prefix;
    unsigned long long *WM = p.wmass + (int64_t)b * nseg * kSegWaves;   // nucleus mass of each wave's ids
    if constexpr (PASS == 4) {
        unsigned long long wm = 0;
        for_tiles([&](int t, const float (&v)[4]) {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const float ev = __builtin_amdgcn_exp2f((v[e] - mx) * kT);
                wm += masked(valid(t) & (__float_as_uint(ev) >= theta), fixed_mass(ev));
            }
        });
        for (int o = 32; o > 0; o >>= 1) {
            const uint32_t lo = __shfl_xor((uint32_t)wm, o), hi = __shfl_xor((uint32_t)(wm >> 32), o);
            wm += ((unsigned long long)hi << 32) | lo;
        }
        if (lane == 0) WM[seg * kSegWaves + wave] = wm;
        return;
    }
    if constexpr (PASS == 5) {
        const unsigned long long M = st.all ? st.total : st.mass;
        const uint64_t r24 =
            splitmix64(rng_key(p.seeds[b], 1ull << 33) + 2ull * (uint64_t)p.step[b] + (uint64_t)p.slot) >> 40;
        const unsigned long long tsel = __umul64hi(r24 << 40, M);
        // the waves before this one, in id order
        const int gw = seg * kSegWaves + wave;
        unsigned long long run = 0;
        for (int w = 0; w < gw; ++w) run += WM[w];
        const unsigned long long wm = WM[gw];
        if (wm == 0 || tsel < run || tsel >= run + wm) return;
        for (int t = 0; t < nt; ++t) {
            float v[4];
            load4(t, v);
            unsigned long long m4[4], loc = 0;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const float ev = __builtin_amdgcn_exp2f((v[e] - mx) * kT);
                m4[e] = masked(valid(t) & (__float_as_uint(ev) >= theta), fixed_mass(ev));
                loc += m4[e];
            }
            unsigned long long inc = loc;
            for (int d = 1; d < 64; d <<= 1) {
                const unsigned long long o = shfl_up_u64(inc, d);
                if (lane >= d) inc += o;
            }
            const unsigned long long excl = run + inc - loc;
            if (loc > 0 && excl <= tsel && tsel < excl + loc) {
                unsigned long long r = excl;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    r += m4[e];
                    if (m4[e] > 0 && r > tsel) {
                        p.best[b] = (1ull << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)(w0 + t * 256 + 4 * lane + e));
                        break;
                    }
                }
            }
            run += __shfl(inc, 63);
            if (run > tsel) break;
        }
    }
}

// Rows split over the segmented kernels: about 256 workgroups in all, 4 to 32 per row.
int sample_segments(int B) {
    int n = 256 / (B > 0 ? B : 1);
    return n < 4 ? 4 : (n > 32 ? 32 : n);
}

void launch_sample(const SampleParams &p, hipStream_t s) {
    if (p.top_k > 0 || p.rep_penalty != 1.f) {
        hipLaunchKernelGGL(k_sample<true>, dim3(p.B), dim3(kSampThreads), 0, s, p);
    } else if (p.hist && p.nseg > 0) {
        SampleParams q = p;
        // segments of whole 1024-id blocks (four waves of 256-id sub-tiles)
        q.seg_len = ((p.V + p.nseg * 1024 - 1) / (p.nseg * 1024)) * 1024;
        const dim3 grid(p.B * p.nseg), block(kSegThreads);
        hipLaunchKernelGGL(k_sample_seg<0>, grid, block, 0, s, q);
        hipLaunchKernelGGL(k_sample_seg<1>, grid, block, 0, s, q);
        hipLaunchKernelGGL(k_sample_seg<2>, grid, block, 0, s, q);
        hipLaunchKernelGGL(k_sample_seg<3>, grid, block, 0, s, q);
        hipLaunchKernelGGL(k_sample_seg<4>, grid, block, 0, s, q);
        hipLaunchKernelGGL(k_sample_seg<5>, grid, block, 0, s, q);
    } else {
        hipLaunchKernelGGL(k_sample<false>, dim3(p.B), dim3(kSampThreads), 0, s, p);
    }
}

}  // namespace pipo
