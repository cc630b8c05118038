// OPD training targets (App. C): per position t of a rolled-out trajectory,
// the sampled reverse-KL term d_t = log p_s(y_t) - log p_t(y_t) and the
// confidence head's target alpha_t = exp(-max(d_t, 0)), from the student's
// and the teacher's logit rows; the teacher row of each position comes from
// PAD compaction (the teacher ran on the trajectory with its PADs removed).
//
// k_opd_rows: one workgroup scans the PAD mask (row = non-PAD count up to
//   and including t, minus one).
// k_opd: one workgroup per position streams its student row and its teacher
//   row once, with a running max and a rescaled exp-sum per thread (online
//   log-sum-exp), float4 loads; the two log-sum-exps and the label's logits
//   give d_t and alpha_t.  HBM-bound: 2 V fp32 per position.
// k_opd_sums: one workgroup adds d over even and odd scored positions in
//   double, in a fixed order.
#include "device_common.h"
#include "pipo.h"

namespace pipo {

constexpr int kOpdThreads = 256;

__global__ __launch_bounds__(1024) void k_opd_rows(const int32_t *tokens, int T, int32_t pad_id, int32_t *rows) {
    __shared__ int s_wave[16];
    __shared__ int s_base;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    if (tid == 0) s_base = 0;
    __syncthreads();
    for (int t0 = 0; t0 < T; t0 += 1024) {
        const int t = t0 + tid;
        const int keep = (t < T && tokens[t] != pad_id) ? 1 : 0;
        int inc = keep;   // inclusive scan inside the wave
        for (int d = 1; d < 64; d <<= 1) {
            const int o = __shfl_up(inc, d);
            if (lane >= d) inc += o;
        }
        if (lane == 63) s_wave[wave] = inc;
        __syncthreads();
        int before = s_base;
        for (int w = 0; w < wave; ++w) before += s_wave[w];
        if (t < T) rows[t] = before + inc - 1;
        __syncthreads();
        if (tid == 1023) s_base = before + inc;
        __syncthreads();
    }
}

// running (max, sum of exp(x - max)) of a stream, merged pairwise; the
// exponentials are the hardware exp2 of (x - max) log2(e)
constexpr float kLog2e = 1.4426950408889634f;
struct Lse { float m, s; };
__device__ __forceinline__ float exp_e(float x) { return __builtin_amdgcn_exp2f(x * kLog2e); }
__device__ __forceinline__ Lse lse_add4(Lse a, f32x4 u) {
    const float m4 = fmaxf(fmaxf(u[0], u[1]), fmaxf(u[2], u[3]));
    if (m4 > a.m) {   // rescale the running sum to the new max (exp(-inf) = 0 at the start)
        a.s *= exp_e(a.m - m4);
        a.m = m4;
    }
    a.s += (exp_e(u[0] - a.m) + exp_e(u[1] - a.m)) + (exp_e(u[2] - a.m) + exp_e(u[3] - a.m));
    return a;
}
__device__ __forceinline__ Lse lse_merge(Lse a, Lse b) {
    if (b.m == -INFINITY) return a;
    if (a.m == -INFINITY) return b;
    const float m = fmaxf(a.m, b.m);
    return Lse{m, a.s * exp_e(a.m - m) + b.s * exp_e(b.m - m)};
}

// Four consecutive logits as floats: fp32 rows (one 16-byte load) or bf16
// rows (one 8-byte load, widened exactly).
template <typename L> struct Logit4;
template <> struct Logit4<float> {
    static __device__ __forceinline__ f32x4 load(const float *row, int i) {
        return __builtin_nontemporal_load((const f32x4 *)row + i);
    }
    static __device__ __forceinline__ float at(const float *row, int y) { return row[y]; }
};
template <> struct Logit4<uint16_t> {
    static __device__ __forceinline__ f32x4 load(const uint16_t *row, int i) {
        const u32x2 w = __builtin_nontemporal_load((const u32x2 *)row + i);
        return f32x4{bf_lo(w[0]), bf_hi(w[0]), bf_lo(w[1]), bf_hi(w[1])};
    }
    static __device__ __forceinline__ float at(const uint16_t *row, int y) {
        return __uint_as_float((uint32_t)row[y] << 16);
    }
};

template <typename L>
__global__ __launch_bounds__(kOpdThreads) void k_opd(const L *ls, const L *lt, const int32_t *rows,
                                                     const int32_t *labels, int T, int V, int Tt, float *kl,
                                                     float *alpha) {
    __shared__ Lse s_red[2][kOpdThreads / 64];
    const int t = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int y = labels[t];
    if (y < 0) {   // not scored (uniform branch: every thread of the workgroup leaves)
        if (tid == 0) { kl[t] = 0.f; alpha[t] = 1.f; }
        return;
    }
    const int r = rows ? rows[t] : t;
    if (r < 0 || r >= Tt || y >= V) {   // no teacher row, or no such token: flagged, not clamped
        if (tid == 0) { kl[t] = __builtin_nanf(""); alpha[t] = __builtin_nanf(""); }
        return;
    }
    const L *rs = ls + (int64_t)t * V;
    const L *rt = lt + (int64_t)r * V;
    Lse a{-INFINITY, 0.f}, b{-INFINITY, 0.f};
    const int V4 = V >> 2;
    for (int i = tid; i < V4; i += kOpdThreads) {
        a = lse_add4(a, Logit4<L>::load(rs, i));
        b = lse_add4(b, Logit4<L>::load(rt, i));
    }
    for (int o = 32; o > 0; o >>= 1) {
        a = lse_merge(a, Lse{__shfl_xor(a.m, o), __shfl_xor(a.s, o)});
        b = lse_merge(b, Lse{__shfl_xor(b.m, o), __shfl_xor(b.s, o)});
    }
    if (lane == 0) { s_red[0][wave] = a; s_red[1][wave] = b; }
    __syncthreads();
    if (tid == 0) {
        Lse A = s_red[0][0], Bt = s_red[1][0];
        for (int w = 1; w < kOpdThreads / 64; ++w) {
            A = lse_merge(A, s_red[0][w]);
            Bt = lse_merge(Bt, s_red[1][w]);
        }
        const float lps = Logit4<L>::at(rs, y) - (A.m + logf(A.s));
        const float lpt = Logit4<L>::at(rt, y) - (Bt.m + logf(Bt.s));
        const float d = lps - lpt;
        kl[t] = d;
        alpha[t] = expf(-fmaxf(d, 0.f));
    }
}

__global__ __launch_bounds__(1024) void k_opd_sums(const float *kl, const int32_t *labels, int T, double *sums) {
    __shared__ double s_v[4][16];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    double v[4] = {0.0, 0.0, 0.0, 0.0};
    for (int t = tid; t < T; t += 1024) {
        if (labels[t] < 0) continue;
        const int par = t & 1;
        v[2 * par] += (double)kl[t];
        v[2 * par + 1] += 1.0;
    }
    for (int k = 0; k < 4; ++k) {
        double x = v[k];
        for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o);
        if (lane == 0) s_v[k][wave] = x;
    }
    __syncthreads();
    if (tid < 4) {
        double x = 0.0;
        for (int w = 0; w < 16; ++w) x += s_v[tid][w];
        sums[tid] = x;
    }
}

}  // namespace pipo

using namespace pipo;

extern "C" int pipo_opd_teacher_rows(const int32_t *d_tokens, int32_t T, int32_t pad_id, int32_t *d_rows,
                                     void *stream) {
    if (!d_tokens || !d_rows || T < 0) return PIPO_EINVAL;
    if (T == 0) return PIPO_OK;
    hipLaunchKernelGGL(k_opd_rows, dim3(1), dim3(1024), 0, (hipStream_t)stream, d_tokens, T, pad_id, d_rows);
    return hipGetLastError() == hipSuccess ? PIPO_OK : PIPO_EHIP;
}

template <typename L>
static int opd_targets(int32_t T, int32_t V, const L *d_logits_s, const L *d_logits_t, int32_t Tt,
                       const int32_t *d_teacher_rows, const int32_t *d_labels, float *d_kl, float *d_alpha,
                       double *d_sums, void *stream) {
    if (T < 0 || V < 1 || Tt < 1 || V % 4) return PIPO_EINVAL;
    hipStream_t s = (hipStream_t)stream;
    if (T > 0) {   // an empty chunk needs no arrays (its sums are zero)
        if (!d_logits_s || !d_logits_t || !d_labels || !d_kl || !d_alpha) return PIPO_EINVAL;
        if (((uintptr_t)d_logits_s | (uintptr_t)d_logits_t) & (4 * sizeof(L) - 1)) return PIPO_EINVAL;   // 4-value rows
        hipLaunchKernelGGL(k_opd<L>, dim3(T), dim3(kOpdThreads), 0, s, d_logits_s, d_logits_t, d_teacher_rows,
                           d_labels, T, V, Tt, d_kl, d_alpha);
    }
    if (d_sums) hipLaunchKernelGGL(k_opd_sums, dim3(1), dim3(1024), 0, s, d_kl, d_labels, T, d_sums);
    return hipGetLastError() == hipSuccess ? PIPO_OK : PIPO_EHIP;
}

extern "C" int pipo_opd_targets(int32_t T, int32_t V, const float *d_logits_s, const float *d_logits_t, int32_t Tt,
                                const int32_t *d_teacher_rows, const int32_t *d_labels, float *d_kl, float *d_alpha,
                                double *d_sums, void *stream) {
    return opd_targets<float>(T, V, d_logits_s, d_logits_t, Tt, d_teacher_rows, d_labels, d_kl, d_alpha, d_sums,
                              stream);
}

extern "C" int pipo_opd_targets_bf16(int32_t T, int32_t V, const uint16_t *d_logits_s, const uint16_t *d_logits_t,
                                     int32_t Tt, const int32_t *d_teacher_rows, const int32_t *d_labels, float *d_kl,
                                     float *d_alpha, double *d_sums, void *stream) {
    return opd_targets<uint16_t>(T, V, d_logits_s, d_logits_t, Tt, d_teacher_rows, d_labels, d_kl, d_alpha, d_sums,
                                 stream);
}
