// Launch interfaces of the gfx950 kernels (host side).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pipo {

// ----------------------------------------------------------------------------
// Weight-streaming skinny GEMM for the decode step:  Y^T[N][B] = W[N][K] X^T.
// W is tiled (16x32 tiles, see device_common.h), X is produced on the fly by
// the prologue into LDS as a bf16 pair (hi + lo, about 16 significant bits),
// B <= 64.
// ----------------------------------------------------------------------------
enum GemvPro : int {
    PRO_NORM = 0,   // X = bf16(RMSNorm(x) * gain): x fp32 [B][K], sum-of-squares parts
    PRO_F32  = 1,   // X = xf, fp32 [B][K]
    PRO_PAIR = 2,   // X = [E[a]; E[b]] for int32 pairs [B][2] (pair-in compressor)
    PRO_MTP  = 3,   // X = [RMSNorm(h_b) g1; RMSNorm(E[tok]) g2], tok from an argmax key
    PRO_CAT  = 4,   // X = RMSNorm([x; x2]) * gain over 2H (one scale): the MLP confidence head
};
// Larger batches: a preparation kernel writes X (RMSNorm and gain applied) as
// bf16 planes hi + lo [B][K] (GemvParams::xh / xl) and the GEMV streams its
// B operands from them (cached in L2) next to the weight tiles.
enum GemvEpi : int {
    EPI_STORE  = 0,  // out fp32 [B][N] = acc (+ bias); sum-of-squares parts
    EPI_RESID  = 1,  // out fp32 [B][N] += acc; sum-of-squares parts
    EPI_SWIGLU = 2,  // act fp32 [B][N/2] = SiLU(gate) * up (gate/up strip-interleaved)
    EPI_QKV    = 3,  // RoPE q,k; q fp32 [B][n_q][d]; k, v appended to the bf16 KV cache
    EPI_LOGITS = 4,  // logits fp32 [B][N]; optional argmax key per row (greedy)
    EPI_SILU   = 5,  // act fp32 [B][N] = SiLU(acc)
};

struct GemvParams {
    const uint16_t *W;          // tiled [N][K]
    int N, K, B;
    int wg_cap;                 // workgroups of the batch-1 kernel, each taking every wg_cap-th
                                // strip group (0: one workgroup per strip group)
    // prologue
    const float *x; const float *xf; const float *ss; int nss; const float *gain;
    const float *x2; const float *ss2;   // PRO_CAT: second half [B][H] and its sum-of-squares parts
    const float *gain2; float eps; const int32_t *pairs; const uint16_t *embed; int H; int vocab;
    const uint64_t *tokkey;
    // epilogue
    float *out; const float *bias; float *ss_out; float *act;
    float *q; uint16_t *kc; uint16_t *vc; const int32_t *pos;
    const float *rope_cos; const float *rope_sin;
    int n_q, n_kv, d, lmax_pad;   // KV geometry of this layer
    int64_t kv_bstride;           // elements between consecutive sequences' caches
    uint64_t *best;               // argmax keys [B] (EPI_LOGITS; NULL: none)
    uint16_t *xh, *xl;            // X planes workspace, [B][K] bf16 each (large batches)
    float *part; int64_t part_cap;  // k-range partial sums workspace (floats): [range][B][N], or
                                    // [range][strip][B][16] above 16 sequences (part_index in gemv.hip)
    int ksplit;                   // k-ranges (set by launch_gemv)
    int *deferred;                // EPI_QKV: if not NULL and K is cut into 2..kAttnFusedRanges ranges,
                                  // the range sum, RoPE and KV append are left to the decode attention
                                  // and *deferred is set to the number of ranges (it stays 0 when the
                                  // epilogue ran)
    int krt;                      // k-tiles per range of the k-range kernel (set by launch_gemv)
    int xseg;                     // 2048-column segments per row of the X planes (set by launch_gemv)
};
// Returns 0, or -1 (nothing launched) for a (pro, epi) pair without an
// instantiation.
int launch_gemv(const GemvParams &p, int pro, int epi, hipStream_t s);
// Profiling of the next launch_gemv on this thread: with `pending` set, the
// call records `start` / `stop` around its kernels (the batch-1 kernel through
// hipExtLaunchKernelGGL, so the interval is the kernel's own execution) and
// clears `pending`.
struct GemvTiming { hipEvent_t start, stop; bool pending; };
extern thread_local GemvTiming g_gemv_timing;
int gemv_num_groups(int N);

// ----------------------------------------------------------------------------
// Split-K grouped-query flash-decode over the latent KV cache.
// ----------------------------------------------------------------------------
// k-ranges of the QKV GEMV whose sum the decode attention takes over (one
// round trip of partial loads in its prologue)
constexpr int kAttnFusedRanges = 4;
// splits == kAttnWgSplits: one workgroup per (sequence, KV group) whose waves
// are the splits, merged in LDS (no k_attn_merge launch); four (4B at batch
// 32: 9.20 ms per pair step against 9.26 with eight, one wave per SIMD)
constexpr int kAttnWgSplits = 4;
// the XCD-local merge (AttnDecodeParams::xl_ctr) is used up to this many
// splits: one wave merges them twelve at a time, and past two rounds of
// requests a merge launch of its own finishes sooner
constexpr int kAttnXcdMergeMaxSplits = 24;

struct AttnDecodeParams {
    const float *q;             // fp32 [B][n_q][d]
    // with qkv_part: the QKV GEMV left its k-range partial sums [ksplit][B][nqkv]
    // (rows in its strip order); the attention adds them, applies RoPE to q and
    // k and appends k, v at pos (instead of reading q)
    const float *qkv_part; int ksplit, nqkv;
    const float *rope_cos, *rope_sin;
    const uint16_t *kc, *vc;    // this layer's caches
    int64_t kv_bstride;
    const int32_t *pos;         // [B]: attend to keys 0..pos[b]
    int B, n_q, n_kv, d, lmax_pad, splits;
    float *part;                // [B][n_q][splits][attn_part_stride(d)]: o[d], m, l, padding
    float *out;                 // fp32 [B][n_q * d]
    // not NULL: the splits of one (sequence, KV group) run on one XCD (the
    // grid is laid out for workgroup i to run on XCD i mod 8) and the last
    // one to finish merges them through that XCD's L2; one counter per
    // (sequence, KV group), left at zero
    int *xl_ctr;
};
// floats per (head, split) record of the attention partials: o, m, l and
// padding to a multiple of 128 bytes, so that no two records share a cache line
constexpr int attn_part_stride(int d) { return d + 32; }
void launch_attn_decode(const AttnDecodeParams &p, hipStream_t s);
// Whether workgroup i of a launch runs on XCD i mod 8 (what an XCD-local merge
// needs): a probe grid records each workgroup's XCD; *ok set from that.
hipError_t probe_xcd_round_robin(hipStream_t s, bool *ok);

// ----------------------------------------------------------------------------
// Heads: confidence gate, top-p sampler.
// ----------------------------------------------------------------------------
struct GateParams {
    const float *hb, *hd; const float *ss_b, *ss_d; int nss_b, nss_d;
    const float *w_conf, *g_conf; int H; float eps, tau;
    const float *conf_h, *conf_w2;   // MLP confidence head: s = conf_w2 . conf_h[b] (H each); NULL: one linear
    uint64_t *best_b, *best_d; int32_t pad_id;
    void *out;                  // pipo_pair [B]
    int32_t *pairs, *pos, *step; int advance;
    int B;
    uint32_t *seen; int seen_words;   // non-NULL: the input pair's tokens join the penalised-token bitmap
    int V;
};
void launch_gate(const GateParams &p, hipStream_t s);

// Regular decoding (no compressor, one token per position and step).
void launch_embed_step(const int32_t *pairs, const uint16_t *embed, int H, int V, float *x, float *ss, int B,
                       int both, hipStream_t s);
void launch_regular_out(uint64_t *best, int32_t *out_tok, int32_t *pairs, int32_t pad_id, int32_t *pos,
                        int32_t *step, int advance, int B, uint32_t *seen, int seen_words, int V, hipStream_t s);
// Penalised-token bitmaps [B][seen_words] (bit t of word t/32: token t):
// set the bit of every prompt token (ids outside [0, V) are skipped).
// `ntok` (device [B], or NULL: n each) bounds each sequence's prompt inside
// its row of stride n.
void launch_seen_mark(const int32_t *tokens, int n, const int32_t *ntok, int B, int V, uint32_t *seen, int seen_words,
                      hipStream_t s);

// State of the segmented top-p selection after each pass (one per row).
struct SampState {
    uint32_t prefix;             // the e-value bits chosen so far
    int all;                     // no value reached top_p (rounding): every token is in the nucleus
    unsigned long long above, mass, total;   // fixed-point masses above the prefix, of the nucleus, of the row
};
struct SampleParams {
    const float *logits; int V; int B;
    float temperature, top_p;
    const uint64_t *seeds; const int32_t *step; int slot;
    uint64_t *best;
    // the evaluation sampler, when top_k > 0 or rep_penalty != 1
    int top_k; float rep_penalty;
    const uint32_t *seen; int seen_words;   // penalised tokens per sequence
    const int32_t *pairs; int32_t pad_id;   // the step's input pair, also penalised (NULL: none)
    const uint64_t *extra_key;              // argmax key of one more penalised token (NULL: none)
    float *pen;                             // workspace [B][V]: the penalised logits
    // temperature + top-p split over nseg workgroups per row (NULL hist: one
    // workgroup per row); best[b] must hold the row's argmax key on entry
    int nseg, seg_len;                      // seg_len is set by launch_sample
    unsigned long long *hist;               // [B][4][nseg][256] per-segment histograms
    SampState *state;                       // [5][B] state after each pass
    unsigned long long *wmass;              // [B][nseg][4] nucleus mass per wave
};
void launch_sample(const SampleParams &p, hipStream_t s);
int sample_segments(int B);

// ----------------------------------------------------------------------------
// Initialisation: R-spec weights into packed layouts, RoPE table.
// ----------------------------------------------------------------------------
enum RowPerm : int { PERM_NONE = 0, PERM_QK = 1, PERM_GATEUP = 2 };
// Fill a tiled [N][K] bf16 matrix: packed row r holds logical row L(r) of
// tensor `tid` (rows [row_lo, row_hi) of the packed matrix); `perm` and
// `half` describe L (see init.hip).
void launch_init_tiled(uint16_t *dst, int64_t N, int64_t K, int64_t row_lo, int64_t row_hi,
                       uint64_t seed, uint64_t tid, int perm, int half, int64_t tid_row0,
                       uint64_t tid2, hipStream_t s);
void launch_init_vec(float *dst, int64_t n, uint64_t seed, uint64_t tid, int kind, hipStream_t s);
void launch_rope_table(float *cos_t, float *sin_t, int lmax, int d, double base, hipStream_t s);
void launch_read_tiled(const uint16_t *src, int64_t N, int64_t K, int64_t start, int64_t count,
                       int perm, int half, int64_t row_base, int64_t rows_total,
                       uint16_t *dst, hipStream_t s);
void launch_fill_u32(uint32_t *p, uint32_t v, int64_t n, hipStream_t s);
void launch_copy_bytes(void *dst, const void *src, int64_t n, hipStream_t s);

// ----------------------------------------------------------------------------
// Prefill: gather, RMSNorm, MFMA GEMM, causal flash attention, last-row pick.
// ----------------------------------------------------------------------------
struct PrefillGeom {
    int B;           // sequences
    int c0, clen;    // chunk start latent and latents in this chunk (the longest sequence's)
    int mpad;        // per-sequence row stride (clen rounded up to 16)
    int n_tok;       // row stride of the token array, and every prompt's length when ntok is NULL
    const int32_t *ntok;   // per-sequence prompt lengths [B] (ragged batch), or NULL
    int tok_per_pos;       // prompt tokens per position: 2 (pairs), 1 (regular decoding)
};
// Prompt tokens of sequence b.
__device__ __forceinline__ int seq_tokens(const PrefillGeom &g, int b) { return g.ntok ? g.ntok[b] : g.n_tok; }
void launch_gather_pairs(const int32_t *tokens, const uint16_t *embed, int H, int V, int pad_id,
                         const PrefillGeom &g, uint16_t *xin, hipStream_t s);
void launch_gather_pair_sum(const int32_t *tokens, const uint16_t *embed, int H, int V, int pad_id,
                            const PrefillGeom &g, float *x, hipStream_t s);
void launch_mtp_rows(const float *xb, const int32_t *tokens, const uint16_t *embed, const float *gh, const float *ge,
                     int H, int V, int pad_id, float eps, const PrefillGeom &g, int M, uint16_t *xh, uint16_t *xl,
                     hipStream_t s);
void launch_gather_tokens(const int32_t *tokens, const uint16_t *embed, int H, int V, int pad_id,
                          const PrefillGeom &g, float *x, hipStream_t s);
void launch_rmsnorm_tiled(const float *x, const float *gain, int H, float eps, int M,
                          uint16_t *xn_hi, uint16_t *xn_lo, hipStream_t s);
// Activations of the prefill GEMMs are a pair of tiled bf16 planes, hi and lo
// (x ~= hi + lo); Xlo == NULL means the activation is exact in bf16.
struct GemmParams {
    const uint16_t *W; const uint16_t *X; const uint16_t *Xlo;   // tiled [N][K], tiled [M][K] x2
    int N, K, M;
    int epi;                                // EPI_STORE (bias), EPI_RESID, EPI_SWIGLU, EPI_QKV, EPI_SILU
    PrefillGeom g;
    float *out; const float *bias; uint16_t *act_hi, *act_lo;
    uint16_t *q, *q_lo;                     // EPI_QKV: the query as hi and lo planes
    uint16_t *kc; uint16_t *vc;
    const float *rope_cos; const float *rope_sin;
    int n_q, n_kv, d, lmax_pad; int64_t kv_bstride;
};
void launch_gemm(const GemmParams &p, hipStream_t s);
struct AttnPrefillParams {
    const uint16_t *q, *q_lo;   // bf16 [B][n_q][mpad][d] each: the query as hi + lo
    const uint16_t *kc, *vc; int64_t kv_bstride;
    PrefillGeom g;
    int n_q, n_kv, d, lmax_pad;
    uint16_t *out_hi, *out_lo;  // tiled [B*mpad][n_q*d], hi and lo planes
};
void launch_attn_prefill(const AttnPrefillParams &p, hipStream_t s);
// After a chunk: every sequence whose last position (ceil(n_b / 2) - 1, or
// n_b - 1 with `regular`) lies in the chunk takes that row as its step state.
void launch_pick_last(const float *x, int H, const PrefillGeom &g, float *xdec, float *ss,
                      int32_t *pos, int32_t *step, int regular, hipStream_t s);

}  // namespace pipo
