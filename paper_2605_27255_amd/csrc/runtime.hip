// Host runtime behind the C ABI: owns device memory, builds the per-step
// launch sequence, drives the chunked prefill and replays the decode step as
// a HIP graph.
#include <hip/hip_runtime.h>
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>
#include <algorithm>
#include <mutex>
#include <string>
#include <vector>

#include "pipo.h"
#include "kernels.h"

using namespace pipo;

namespace {

thread_local std::string g_init_error = "no error";

int64_t round_up(int64_t v, int64_t m) { return (v + m - 1) / m * m; }

struct LayerW {
    uint16_t *wqkv, *wo, *wgu, *wdown;
    float *g_attn, *g_ffn;
};

struct Arena {
    char *base = nullptr;
    size_t used = 0, cap = 0;
    template <class T>
    T *take(int64_t n) {
        size_t bytes = (size_t)round_up((int64_t)(n * sizeof(T)), 256);
        T *p = (T *)(base + used);
        used += bytes;
        return p;
    }
};

}  // namespace

struct pipo_ctx {
    pipo_config cfg;
    uint64_t seed;
    int H, F, V, nq, nkv, d, L, qdim, kvdim, nqkv, pad_id, Bmax, lmax_pad, chunk;
    int64_t kv_bstride;    // elements between sequences in one layer's K (or V) cache
    std::string err = "no error";

    char *wmem = nullptr, *amem = nullptr;
    uint16_t *embed, *w_comp, *w_fc;
    float *b_comp, *w_conf, *g_final, *g_mtp_h, *g_mtp_e, *g_mtp_o, *g_conf;
    std::vector<LayerW> layers;
    uint16_t *kc, *vc;
    // App. B heads (pipo_config.heads): MLP compressor, MTP decoder layer with
    // its KV cache, MLP confidence head
    int heads = 0;
    uint16_t *comp_w1 = nullptr, *comp_w2 = nullptr, *conf_w1 = nullptr;
    float *conf_w2 = nullptr;
    LayerW mtp{};
    uint16_t *kc_mtp = nullptr, *vc_mtp = nullptr;
    float *rope_cos, *rope_sin;

    // decode state and activations
    float *x, *ss_x, *hd, *ss_hd, *logits_b, *logits_d, *apart;
    float *qbuf, *attn_out, *act;
    uint16_t *xh, *xl;    // decode GEMV input planes for larger batches [Bmax][Kmax]
    float *gpart; int64_t gpart_cap;   // decode GEMV k-range partial sums
    int n_cu;             // compute units: workgroups of the batch-1 GEMV
    int32_t *xl_ctr = nullptr;   // decode attention: per (sequence, KV group) split counters, kept at zero
    bool xl_merge = false;       // merge the attention splits on their XCD (placement probed at init)
    int dev = 0;          // the device the context lives on
    void *scratch = nullptr;   // that device's address of the static scratch (pipo_decode_step_noalloc)
    uint64_t *best_b, *best_d, *seeds;
    int32_t *pairs, *pos, *step;
    uint32_t *seen; int seen_words;   // penalised-token bitmap per sequence (evaluation sampler)
    float *pen;                       // penalised logits [Bmax][V] (evaluation sampler workspace)
    unsigned long long *samp_hist, *samp_wmass;   // segmented top-p workspace: histograms, wave masses
    SampState *samp_state;
    pipo_pair *out;
    // prefill activations
    uint16_t *p_xin, *p_xn, *p_xn_lo, *p_q, *p_q_lo, *p_o, *p_o_lo, *p_act, *p_act_lo;
    float *p_x;

    uint64_t *h_seeds = nullptr;     // pinned staging for sampler seeds
    hipEvent_t seeds_done = nullptr;
    int32_t *h_lens = nullptr;       // pinned staging for the prompt lengths of a ragged batch
    hipEvent_t lens_done = nullptr;
    int32_t *ntok = nullptr;         // device: prompt lengths of the last ragged prefill [Bmax]
    hipStream_t cap_stream = nullptr;

    int batch = 0, len = 0;
    bool prefilled = false;
    bool regular = false;           // the last prefill was regular decoding
    int32_t *out_tok = nullptr;     // regular decoding: selected token per sequence
    hipGraphExec_t graph_reg = nullptr;
    bool graph_reg_dirty = true;
    float tau = 0.5f, temperature = 0.f, top_p = 1.f;
    int top_k = 0; float rep_penalty = 1.f;
    bool eval_smp = false;          // top-k or repetition penalty in use

    hipGraphExec_t graph = nullptr;
    bool graph_dirty = true;
    bool use_graph = true;
    // PIPO_CHECK=1 in the environment at init: launch eagerly, wait for the
    // stream after every kernel and report the first failure with its site
    bool check = false;
    int enq_rc = PIPO_OK;            // first failure while enqueueing the current call

    // profiling: events around every launch, summed per kernel class
    bool prof_on = false;
    std::vector<hipEvent_t> ev_pool;
    size_t ev_next = 0;
    std::vector<std::pair<int, size_t>> pending;   // (class, index of the start event)
    double prof_ms[PIPO_K_CLASSES] = {};
    int64_t prof_n[PIPO_K_CLASSES] = {};
};

static void check_launch(pipo_ctx *c, hipStream_t s, int cls, int line);

// Launch bracket: record an event before and after a launch when profiling;
// in check mode, wait for the launch and take its error.
// Around one launch_gemv call (gemv = true) the events go to the GEMV
// launcher instead, which records them around its kernels (the batch-1
// kernel times itself, without the gaps an event recorded between two
// launches adds).
struct ProfScope {
    pipo_ctx *c; hipStream_t s; int cls; int line; bool gemv; size_t i0 = 0;
    ProfScope(pipo_ctx *c_, hipStream_t s_, int cls_, int line_, bool gemv_ = false)
        : c(c_), s(s_), cls(cls_), line(line_), gemv(gemv_) {
        if (!c->prof_on) return;
        while (c->ev_pool.size() < c->ev_next + 2) {
            hipEvent_t e;
            if (hipEventCreate(&e) != hipSuccess) { c->prof_on = false; return; }
            c->ev_pool.push_back(e);
        }
        i0 = c->ev_next;
        c->ev_next += 2;
        if (gemv) g_gemv_timing = GemvTiming{c->ev_pool[i0], c->ev_pool[i0 + 1], true};
        else hipEventRecord(c->ev_pool[i0], s);
    }
    ~ProfScope() {
        if (c->check) check_launch(c, s, cls, line);
        if (!c->prof_on) return;
        if (!gemv) {
            hipEventRecord(c->ev_pool[i0 + 1], s);
        } else if (g_gemv_timing.pending) {   // nothing was launched: an empty interval
            g_gemv_timing.pending = false;
            hipEventRecord(c->ev_pool[i0], s);
            hipEventRecord(c->ev_pool[i0 + 1], s);
        }
        c->pending.push_back({cls, i0});
    }
};
#define PROF_CAT2(a, b) a##b
#define PROF_CAT(a, b) PROF_CAT2(a, b)
#define PROF(cls) ProfScope PROF_CAT(prof_scope_, __LINE__)(c, s, cls, __LINE__)
#define PROF_GEMV(cls) ProfScope PROF_CAT(prof_scope_, __LINE__)(c, s, cls, __LINE__, true)

static int fail(pipo_ctx *c, int code, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    if (c) c->err = buf;
    else g_init_error = buf;
    return code;
}

static void check_launch(pipo_ctx *c, hipStream_t s, int cls, int line) {
    hipError_t e = hipGetLastError();
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e == hipSuccess) e = hipGetLastError();
    if (e != hipSuccess && c->enq_rc == PIPO_OK)
        c->enq_rc = fail(c, PIPO_EHIP, "PIPO_CHECK: kernel of class %d launched at runtime.hip:%d failed: %s", cls,
                         line, hipGetErrorString(e));
}

// launch_gemv; a (prologue, epilogue) pair it has no kernel for is the call's error
static void gemv(pipo_ctx *c, const GemvParams &p, int pro, int epi, hipStream_t s) {
    if (launch_gemv(p, pro, epi, s) != 0 && c->enq_rc == PIPO_OK)
        c->enq_rc = fail(c, PIPO_EINVAL, "no decode GEMV kernel for prologue %d with epilogue %d", pro, epi);
}

#define HIP_TRY(ctx, expr)                                                                     \
    do {                                                                                       \
        hipError_t e_ = (expr);                                                                \
        if (e_ != hipSuccess)                                                                  \
            return fail((ctx), PIPO_EHIP, "%s failed: %s", #expr, hipGetErrorString(e_));     \
    } while (0)

static int check_config(const pipo_config *c) {
    if (!c) return fail(nullptr, PIPO_EINVAL, "config is NULL");
    if (c->n_layers < 0 || c->hidden <= 0 || c->n_q_heads <= 0 || c->n_kv_heads <= 0 || c->ffn <= 0 ||
        c->vocab <= 1)
        return fail(nullptr, PIPO_EINVAL, "non-positive model dimension");
    if (c->hidden % 32 || c->ffn % 32 || c->vocab % 16)
        return fail(nullptr, PIPO_EINVAL, "hidden and ffn must be multiples of 32, vocab of 16");
    if (c->head_dim != 64 && c->head_dim != 128) return fail(nullptr, PIPO_EINVAL, "head_dim must be 64 or 128");
    if (c->n_q_heads % c->n_kv_heads || c->n_q_heads / c->n_kv_heads > 16)
        return fail(nullptr, PIPO_EINVAL, "n_q_heads must be a multiple of n_kv_heads, at most 16x");
    if ((c->n_q_heads * c->head_dim) % 32) return fail(nullptr, PIPO_EINVAL, "n_q_heads*head_dim % 32 != 0");
    if (c->max_batch < 1 || c->max_batch > 64) return fail(nullptr, PIPO_EINVAL, "max_batch must be in [1, 64]");
    if (c->max_latent < 1 || c->prefill_chunk < 1) return fail(nullptr, PIPO_EINVAL, "max_latent and prefill_chunk must be >= 1");
    if (c->pad_id < -1 || c->pad_id >= c->vocab) return fail(nullptr, PIPO_EINVAL, "pad_id out of range");
    if (!(c->rms_eps >= 0.f) || !(c->rope_base > 0.f)) return fail(nullptr, PIPO_EINVAL, "bad rms_eps or rope_base");
    if (c->gain_mode != 0 && c->gain_mode != 1) return fail(nullptr, PIPO_EINVAL, "gain_mode must be 0 or 1");
    if (c->heads & ~(PIPO_HEADS_MLP_COMPRESSOR | PIPO_HEADS_MTP_LAYER | PIPO_HEADS_MLP_CONFIDENCE))
        return fail(nullptr, PIPO_EINVAL, "unknown heads flags 0x%x", (unsigned)c->heads);
    return PIPO_OK;
}

// tensor ids of the weight generator (model-level; per layer 100 + 10 l + slot)
enum { TID_EMBED = 0, TID_WCOMP = 1, TID_BCOMP = 2, TID_WFC = 3, TID_WCONF = 4, TID_GFINAL = 5,
       TID_GMTPH = 6, TID_GMTPE = 7, TID_GMTPO = 8, TID_GCONF = 9, TID_COMPW1 = 10, TID_COMPW2 = 11,
       TID_CONFW1 = 12, TID_CONFW2 = 13 };
static uint64_t layer_tid(int l, int slot) { return 100ull + 10ull * (uint64_t)l + (uint64_t)slot; }
static uint64_t mtp_tid(int slot) { return 90ull + (uint64_t)slot; }   // the MTP head's decoder layer

// ---- scratch of pipo_decode_step_noalloc -----------------------------------
// A file-scope device array, one copy per GPU held until the process ends:
// the decode attention's split partials at its start, then the k-range
// partial sums of the larger-batch GEMVs.  Host code never passes the
// array's name to a kernel (on the host it is only a stand-in); it uses the
// per-device address hipGetSymbolAddress returns, taken once per device at
// context creation with that device current.
constexpr size_t kScratchBytes = size_t(16) << 20;
static __device__ __align__(256) char scratch[kScratchBytes];
constexpr int kMaxDevices = 64;
static std::mutex g_scratch_mu;
static void *g_scratch_addr[kMaxDevices] = {};

static hipError_t scratch_address(int dev, void **out) {
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_addr[dev]) {
        void *ptr = nullptr;
        const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        g_scratch_addr[dev] = ptr;
    }
    *out = g_scratch_addr[dev];
    return hipSuccess;
}

extern "C" int pipo_init_weights(const pipo_config *cfg, uint64_t seed, void *stream, pipo_ctx **out) {
    if (!out) return fail(nullptr, PIPO_EINVAL, "out is NULL");
    *out = nullptr;
    int rc = check_config(cfg);
    if (rc) return rc;
    hipStream_t s = (hipStream_t)stream;
    pipo_ctx *c = new pipo_ctx();
    c->cfg = *cfg;
    c->seed = seed;
    c->H = cfg->hidden; c->F = cfg->ffn; c->V = cfg->vocab; c->nq = cfg->n_q_heads; c->nkv = cfg->n_kv_heads;
    c->d = cfg->head_dim; c->L = cfg->n_layers; c->qdim = c->nq * c->d; c->kvdim = c->nkv * c->d;
    c->nqkv = c->qdim + 2 * c->kvdim; c->pad_id = cfg->pad_id < 0 ? cfg->vocab - 1 : cfg->pad_id;
    c->Bmax = cfg->max_batch;
    // 128 positions of slack: prefill attention stages 64-key blocks that may
    // extend up to 94 positions past the last latent.
    c->lmax_pad = (int)round_up((int64_t)cfg->max_latent + 128, 64);
    c->chunk = cfg->prefill_chunk;
    c->kv_bstride = (int64_t)c->nkv * c->lmax_pad * c->d;
    c->heads = cfg->heads;
    const int H = c->H, F = c->F, V = c->V, B = c->Bmax;

    // ---- weights --------------------------------------------------------
    Arena w;
    for (int pass = 0; pass < 2; ++pass) {
        w.used = 0;
        c->embed = w.take<uint16_t>((int64_t)V * H);
        c->w_comp = w.take<uint16_t>((int64_t)H * 2 * H);
        c->w_fc = w.take<uint16_t>((int64_t)H * 2 * H);
        c->b_comp = w.take<float>(H);
        c->w_conf = w.take<float>(2 * H);
        c->g_final = w.take<float>(H);
        c->g_mtp_h = w.take<float>(H);
        c->g_mtp_e = w.take<float>(H);
        c->g_mtp_o = w.take<float>(H);
        c->g_conf = w.take<float>(2 * H);
        c->layers.assign(c->L, LayerW{});
        auto take_layer = [&](LayerW &l) {
            l.wqkv = w.take<uint16_t>((int64_t)c->nqkv * H);
            l.wo = w.take<uint16_t>((int64_t)H * c->qdim);
            l.wgu = w.take<uint16_t>((int64_t)2 * F * H);
            l.wdown = w.take<uint16_t>((int64_t)H * F);
            l.g_attn = w.take<float>(H);
            l.g_ffn = w.take<float>(H);
        };
        for (auto &l : c->layers) take_layer(l);
        if (c->heads & PIPO_HEADS_MLP_COMPRESSOR) {
            c->comp_w1 = w.take<uint16_t>((int64_t)H * 2 * H);
            c->comp_w2 = w.take<uint16_t>((int64_t)H * H);
        }
        if (c->heads & PIPO_HEADS_MTP_LAYER) take_layer(c->mtp);
        if (c->heads & PIPO_HEADS_MLP_CONFIDENCE) {
            c->conf_w1 = w.take<uint16_t>((int64_t)H * 2 * H);
            c->conf_w2 = w.take<float>(H);
        }
        if (pass == 0) {
            if (hipMalloc(&c->wmem, w.used) != hipSuccess) {
                delete c;
                return fail(nullptr, PIPO_ENOMEM, "weights: hipMalloc of %zu bytes failed", w.used);
            }
            w.base = c->wmem;
        }
    }

    // ---- KV cache, RoPE table, activations ------------------------------
    Arena a;
    const int64_t mcap = (int64_t)B * round_up(c->chunk, 64);   // rows per chunk: ragged batches pad to 64
    const int S_att = 64;
    for (int pass = 0; pass < 2; ++pass) {
        a.used = 0;
        c->kc = a.take<uint16_t>((int64_t)c->L * B * c->kv_bstride);
        c->vc = a.take<uint16_t>((int64_t)c->L * B * c->kv_bstride);
        if (c->heads & PIPO_HEADS_MTP_LAYER) {
            c->kc_mtp = a.take<uint16_t>((int64_t)B * c->kv_bstride);
            c->vc_mtp = a.take<uint16_t>((int64_t)B * c->kv_bstride);
        }
        c->rope_cos = a.take<float>((int64_t)c->lmax_pad * (c->d / 2));
        c->rope_sin = a.take<float>((int64_t)c->lmax_pad * (c->d / 2));
        c->x = a.take<float>((int64_t)B * H);
        c->hd = a.take<float>((int64_t)B * H);
        c->ss_x = a.take<float>((int64_t)B * (H / 16));
        c->ss_hd = a.take<float>((int64_t)B * (H / 16));
        c->logits_b = a.take<float>((int64_t)B * V);
        c->logits_d = a.take<float>((int64_t)B * V);
        c->qbuf = a.take<float>((int64_t)B * c->qdim);
        c->attn_out = a.take<float>((int64_t)B * c->qdim);
        c->act = a.take<float>((int64_t)B * F);
        {
            const int64_t kmax = std::max<int64_t>(std::max<int64_t>(2 * H, F), c->qdim);
            c->xh = a.take<uint16_t>((int64_t)B * kmax);
            c->xl = a.take<uint16_t>((int64_t)B * kmax);
            // k-range partial sums of the larger-batch GEMV: room for 16 ranges
            // of the widest non-vocabulary output
            const int64_t nmax = std::max<int64_t>(std::max<int64_t>(2 * F, c->nqkv), 2 * H);
            c->gpart_cap = 16 * (int64_t)B * nmax;
            c->gpart = a.take<float>(c->gpart_cap);
        }
        c->best_b = a.take<uint64_t>(B);
        c->best_d = a.take<uint64_t>(B);
        c->seeds = a.take<uint64_t>(B);
        c->pairs = a.take<int32_t>(2 * B);
        c->ntok = a.take<int32_t>(B);
        c->seen_words = (V + 31) / 32;
        c->seen = a.take<uint32_t>((int64_t)B * c->seen_words);
        c->pen = a.take<float>((int64_t)B * V);
        // at most 256 workgroups over the rows: sample_segments(B) * B <= 256
        c->samp_hist = a.take<unsigned long long>((int64_t)256 * 4 * 256);
        c->samp_wmass = a.take<unsigned long long>((int64_t)256 * 4);
        c->samp_state = a.take<SampState>((int64_t)5 * B);
        c->pos = a.take<int32_t>(B);
        c->step = a.take<int32_t>(B);
        c->out = a.take<pipo_pair>(B);
        c->out_tok = a.take<int32_t>(B);
        c->apart = a.take<float>((int64_t)B * c->nq * S_att * attn_part_stride(c->d));
        c->xl_ctr = a.take<int32_t>((int64_t)B * c->nkv);
        c->p_xin = a.take<uint16_t>(mcap * 2 * H);
        c->p_x = a.take<float>(mcap * H);
        c->p_xn = a.take<uint16_t>(mcap * H);
        c->p_xn_lo = a.take<uint16_t>(mcap * H);
        c->p_q = a.take<uint16_t>(mcap * c->qdim);
        c->p_q_lo = a.take<uint16_t>(mcap * c->qdim);
        c->p_o = a.take<uint16_t>(mcap * c->qdim);
        c->p_o_lo = a.take<uint16_t>(mcap * c->qdim);
        c->p_act = a.take<uint16_t>(mcap * F);
        c->p_act_lo = a.take<uint16_t>(mcap * F);
        if (pass == 0) {
            if (hipMalloc(&c->amem, a.used) != hipSuccess) {
                hipFree(c->wmem);
                delete c;
                return fail(nullptr, PIPO_ENOMEM, "KV cache and workspaces: hipMalloc of %zu bytes failed", a.used);
            }
            a.base = c->amem;
        }
    }
    pipo_ctx *cc = c;
    auto cleanup_fail = [&](int code) {
        g_init_error = cc->err;
        pipo_free(cc);
        return code;
    };
    // Zero everything once (argmax keys, the KV cache: attention
    // reads whole 32-key tiles and relies on finite values past the length).
    if (hipMemsetAsync(c->amem, 0, a.used, s) != hipSuccess) return cleanup_fail(fail(c, PIPO_EHIP, "memset failed"));

    // ---- generate weights on the device --------------------------------
    const uint64_t sd = seed;
    launch_init_tiled(c->embed, V, H, 0, V, sd, TID_EMBED, PERM_NONE, 0, 0, 0, s);
    launch_init_tiled(c->w_comp, H, 2 * H, 0, H, sd, TID_WCOMP, PERM_NONE, 0, 0, 0, s);
    launch_init_tiled(c->w_fc, H, 2 * H, 0, H, sd, TID_WFC, PERM_NONE, 0, 0, 0, s);
    launch_init_vec(c->b_comp, H, sd, TID_BCOMP, 0, s);
    launch_init_vec(c->w_conf, 2 * H, sd, TID_WCONF, 0, s);
    const int gk = cfg->gain_mode ? 2 : 1;
    launch_init_vec(c->g_final, H, sd, TID_GFINAL, gk, s);
    launch_init_vec(c->g_mtp_h, H, sd, TID_GMTPH, gk, s);
    launch_init_vec(c->g_mtp_e, H, sd, TID_GMTPE, gk, s);
    launch_init_vec(c->g_mtp_o, H, sd, TID_GMTPO, gk, s);
    launch_init_vec(c->g_conf, 2 * H, sd, TID_GCONF, gk, s);
    auto init_layer = [&](LayerW &lw, auto tid) {
        launch_init_tiled(lw.wqkv, c->nqkv, H, 0, c->qdim, sd, tid(0), PERM_QK, c->d / 2, 0, 0, s);
        launch_init_tiled(lw.wqkv, c->nqkv, H, c->qdim, c->qdim + c->kvdim, sd, tid(1), PERM_QK, c->d / 2, 0, 0, s);
        launch_init_tiled(lw.wqkv, c->nqkv, H, c->qdim + c->kvdim, c->nqkv, sd, tid(2), PERM_NONE, 0, 0, 0, s);
        launch_init_tiled(lw.wo, H, c->qdim, 0, H, sd, tid(3), PERM_NONE, 0, 0, 0, s);
        launch_init_tiled(lw.wgu, 2 * F, H, 0, 2 * F, sd, tid(4), PERM_GATEUP, 0, 0, tid(5), s);
        launch_init_tiled(lw.wdown, H, F, 0, H, sd, tid(6), PERM_NONE, 0, 0, 0, s);
        launch_init_vec(lw.g_attn, H, sd, tid(7), gk, s);
        launch_init_vec(lw.g_ffn, H, sd, tid(8), gk, s);
    };
    for (int l = 0; l < c->L; ++l) init_layer(c->layers[l], [l](int slot) { return layer_tid(l, slot); });
    if (c->heads & PIPO_HEADS_MLP_COMPRESSOR) {
        launch_init_tiled(c->comp_w1, H, 2 * H, 0, H, sd, TID_COMPW1, PERM_NONE, 0, 0, 0, s);
        launch_init_tiled(c->comp_w2, H, H, 0, H, sd, TID_COMPW2, PERM_NONE, 0, 0, 0, s);
    }
    if (c->heads & PIPO_HEADS_MTP_LAYER) init_layer(c->mtp, [](int slot) { return mtp_tid(slot); });
    if (c->heads & PIPO_HEADS_MLP_CONFIDENCE) {
        launch_init_tiled(c->conf_w1, H, 2 * H, 0, H, sd, TID_CONFW1, PERM_NONE, 0, 0, 0, s);
        launch_init_vec(c->conf_w2, H, sd, TID_CONFW2, 0, s);
    }
    launch_rope_table(c->rope_cos, c->rope_sin, c->lmax_pad, c->d, (double)cfg->rope_base, s);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return cleanup_fail(fail(c, PIPO_EHIP, "init launch: %s", hipGetErrorString(e)));
    if (hipHostMalloc((void **)&c->h_seeds, sizeof(uint64_t) * B, hipHostMallocDefault) != hipSuccess ||
        hipEventCreateWithFlags(&c->seeds_done, hipEventDisableTiming) != hipSuccess ||
        hipHostMalloc((void **)&c->h_lens, sizeof(int32_t) * B, hipHostMallocDefault) != hipSuccess ||
        hipEventCreateWithFlags(&c->lens_done, hipEventDisableTiming) != hipSuccess ||
        hipStreamCreateWithFlags(&c->cap_stream, hipStreamNonBlocking) != hipSuccess)
        return cleanup_fail(fail(c, PIPO_EHIP, "host staging / event / stream creation failed"));
    e = hipStreamSynchronize(s);
    if (e != hipSuccess) return cleanup_fail(fail(c, PIPO_EHIP, "init: %s", hipGetErrorString(e)));
    {
        int dev = 0, ncu = 0;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || ncu < 1)
            return cleanup_fail(fail(c, PIPO_EHIP, "compute unit count query failed"));
        c->n_cu = ncu;
        // test hook: fewer GEMV workgroups, so small models run several strip groups per workgroup
        const char *wc = getenv("PIPO_GEMV_WG_CAP");
        if (wc && atoi(wc) > 0) c->n_cu = atoi(wc);
        c->dev = dev;
        const hipError_t se = scratch_address(dev, &c->scratch);
        if (se != hipSuccess)
            return cleanup_fail(fail(c, PIPO_EHIP, "scratch address on device %d: %s", dev, hipGetErrorString(se)));
        // PIPO_NO_XCD_MERGE=1: always merge the attention splits in a kernel of their own
        const char *nx = getenv("PIPO_NO_XCD_MERGE");
        bool rr = false;
        if (!(nx && nx[0] == '1')) {
            const hipError_t pe = probe_xcd_round_robin(s, &rr);
            if (pe != hipSuccess)
                return cleanup_fail(fail(c, PIPO_EHIP, "XCD placement probe: %s", hipGetErrorString(pe)));
        }
        c->xl_merge = rr;
    }
    const char *ng = getenv("PIPO_NO_GRAPH");
    const char *ck = getenv("PIPO_CHECK");
    c->check = ck && ck[0] == '1';
    c->use_graph = !(ng && ng[0] == '1') && !c->check;
    *out = c;
    return PIPO_OK;
}

// Key splits of the decode attention: at most two 32-key blocks per split at
// full capacity (both blocks are prefetched), and no more splits than it takes
// to give the machine about 768 waves, three per CU; at most 64 (the merge
// kernel's limit).  (9B at batch 8, 64 (sequence, KV group) pairs and 517
// blocks: 9 to 16 splits took 3.04, 2.86, 2.82, 2.76, 2.97, 2.87 (14) and
// 2.86 ms of attention per pair step: 12 splits, three waves on every CU.)
// Where at most four blocks per split bring the count within the XCD-local
// merge's limit, the limit it is: the merge launch saved outweighs the
// longer splits (4B at batch 1 and 73 blocks: 37 splits and the launch
// 0.430 ms per step, 24 splits merged on their XCD 0.381 ms; 20: 0.388,
// 16: 0.393, 12: 0.415).
static int attn_splits(const pipo_ctx *c, int B) {
    // a workgroup per (sequence, KV group) once they fill every CU: its
    // kAttnWgSplits waves split the keys and merge in LDS, with no merge launch
    if (B * c->nkv >= c->n_cu) return kAttnWgSplits;
    const int blocks = (c->cfg.max_latent + 31) / 32;
    const int cap = (768 + B * c->nkv - 1) / (B * c->nkv);
    int sp = (blocks + 1) / 2;
    if (c->xl_merge && sp > kAttnXcdMergeMaxSplits && blocks <= 4 * kAttnXcdMergeMaxSplits)
        sp = kAttnXcdMergeMaxSplits;
    sp = sp < cap ? sp : cap;
    return sp < 1 ? 1 : (sp > 64 ? 64 : sp);
}

static GemvParams gemv_base(const pipo_ctx *c, int B) {
    GemvParams p{};
    p.B = B; p.eps = c->cfg.rms_eps; p.H = c->H; p.vocab = c->V; p.xh = c->xh; p.xl = c->xl; p.part = c->gpart;
    p.part_cap = c->gpart_cap; p.wg_cap = c->n_cu;
    return p;
}

// One decoder layer (eq. 2) at the current positions over the residual xres
// (with its sum-of-squares parts ssres): a backbone layer, or the MTP head's.
static void enqueue_layer(pipo_ctx *c, const LayerW &lw, uint16_t *kc, uint16_t *vc, float *xres, float *ssres,
                          hipStream_t s) {
    const int B = c->batch, H = c->H;
    const GemvParams base = gemv_base(c, B);
    GemvParams p = base;
    p.W = lw.wqkv; p.N = c->nqkv; p.K = H;
    p.x = xres; p.ss = ssres; p.nss = H / 16; p.gain = lw.g_attn;
    p.q = c->qbuf; p.kc = kc; p.vc = vc; p.pos = c->pos; p.rope_cos = c->rope_cos; p.rope_sin = c->rope_sin;
    p.n_q = c->nq; p.n_kv = c->nkv; p.d = c->d; p.lmax_pad = c->lmax_pad; p.kv_bstride = c->kv_bstride;
    int ranges = 0;      // k-ranges whose sum (and RoPE, KV append) the attention takes over
    p.deferred = (c->nq / c->nkv) * c->d <= 1024 ? &ranges : nullptr;   // the attention stages q in 4 KB of LDS
    { PROF_GEMV(PIPO_K_GEMV_LAYER); gemv(c, p, PRO_NORM, EPI_QKV, s); }

    AttnDecodeParams ap{};
    ap.q = c->qbuf; ap.kc = kc; ap.vc = vc; ap.kv_bstride = c->kv_bstride; ap.pos = c->pos;
    if (ranges > 1) {
        ap.qkv_part = p.part; ap.ksplit = ranges; ap.nqkv = c->nqkv;
        ap.rope_cos = c->rope_cos; ap.rope_sin = c->rope_sin;
    }
    ap.B = B; ap.n_q = c->nq; ap.n_kv = c->nkv; ap.d = c->d; ap.lmax_pad = c->lmax_pad;
    ap.splits = attn_splits(c, B); ap.part = c->apart; ap.out = c->attn_out;
    ap.xl_ctr = c->xl_merge && ap.splits != kAttnWgSplits && ap.splits <= kAttnXcdMergeMaxSplits ? c->xl_ctr : nullptr;
    { PROF(PIPO_K_ATTN_DECODE); launch_attn_decode(ap, s); }

    p = base;
    p.W = lw.wo; p.N = H; p.K = c->qdim; p.xf = c->attn_out; p.out = xres; p.ss_out = ssres;
    { PROF_GEMV(PIPO_K_GEMV_LAYER); gemv(c, p, PRO_F32, EPI_RESID, s); }

    p = base;
    p.W = lw.wgu; p.N = 2 * c->F; p.K = H; p.x = xres; p.ss = ssres; p.nss = H / 16; p.gain = lw.g_ffn;
    p.act = c->act;
    { PROF_GEMV(PIPO_K_GEMV_LAYER); gemv(c, p, PRO_NORM, EPI_SWIGLU, s); }

    p = base;
    p.W = lw.wdown; p.N = H; p.K = c->F; p.xf = c->act; p.out = xres; p.ss_out = ssres;
    { PROF_GEMV(PIPO_K_GEMV_LAYER); gemv(c, p, PRO_F32, EPI_RESID, s); }
}

// The backbone layers of one decode position over the residual in x.
static void enqueue_layers(pipo_ctx *c, hipStream_t s) {
    for (int l = 0; l < c->L; ++l)
        enqueue_layer(c, c->layers[l], c->kc + (int64_t)l * c->Bmax * c->kv_bstride,
                      c->vc + (int64_t)l * c->Bmax * c->kv_bstride, c->x, c->ss_x, s);
}

// Selection of one slot's tokens from `logits` into `best`.  `in_pair`: the
// step's input pair is in c->pairs (a decode step, not a prefill); `extra`:
// the argmax key of one more token the repetition penalty applies to.
static SampleParams sample_params(pipo_ctx *c, const float *logits, int B, int slot, uint64_t *best, bool in_pair,
                                  const uint64_t *extra) {
    SampleParams sp{};
    sp.logits = logits; sp.V = c->V; sp.B = B; sp.temperature = c->temperature; sp.top_p = c->top_p;
    sp.seeds = c->seeds; sp.step = c->step; sp.slot = slot; sp.best = best;
    sp.top_k = c->top_k; sp.rep_penalty = c->rep_penalty;
    sp.nseg = sample_segments(B); sp.hist = c->samp_hist; sp.state = c->samp_state; sp.wmass = c->samp_wmass;
    if (c->eval_smp) {
        sp.seen = c->seen; sp.seen_words = c->seen_words;
        sp.pairs = in_pair ? c->pairs : nullptr; sp.pad_id = c->pad_id;
        sp.extra_key = extra;
        sp.pen = c->pen;
    }
    return sp;
}

// ---------------------------------------------------------------------------
// The heads of a pair step (eqs. 3-6): LM head + selection of the backbone
// token, MTP head, LM head + selection of the draft, confidence gate.
// `nss` is the number of sum-of-squares parts describing x (h_b); `in_pair`:
// a decode step, whose input pair joins the penalised tokens.
static void enqueue_heads(pipo_ctx *c, int B, int nss, int advance, bool in_pair, hipStream_t s) {
    const int H = c->H;
    const bool greedy = c->temperature <= 0.f;
    GemvParams p{};
    p.B = B; p.eps = c->cfg.rms_eps; p.H = H; p.xh = c->xh; p.xl = c->xl; p.part = c->gpart; p.part_cap = c->gpart_cap;
    // LM head #1 on RMSNorm(h_b; g_final)
    p.W = c->embed; p.N = c->V; p.K = H;
    p.x = c->x; p.ss = c->ss_x; p.nss = nss; p.gain = c->g_final;
    p.out = c->logits_b; p.best = c->best_b;   // sampling reads the row max from the key
    { PROF_GEMV(PIPO_K_GEMV_LMHEAD); gemv(c, p, PRO_NORM, EPI_LOGITS, s); }
    if (!greedy) {
        PROF(PIPO_K_SAMPLE);
        launch_sample(sample_params(c, c->logits_b, B, 0, c->best_b, in_pair, nullptr), s);
    }
    // MTP head: W_fc [RMSNorm(h_b; g_mh); RMSNorm(E[b]; g_me)]
    GemvParams m{};
    m.B = B; m.eps = c->cfg.rms_eps; m.H = H; m.vocab = c->V; m.xh = c->xh; m.xl = c->xl; m.part = c->gpart; m.part_cap = c->gpart_cap;
    m.wg_cap = c->n_cu;
    m.W = c->w_fc; m.N = H; m.K = 2 * H;
    m.x = c->x; m.ss = c->ss_x; m.nss = nss; m.gain = c->g_mtp_h; m.gain2 = c->g_mtp_e;
    m.embed = c->embed; m.tokkey = c->best_b;
    m.out = c->hd; m.ss_out = c->ss_hd;
    { PROF_GEMV(PIPO_K_GEMV_SMALL); gemv(c, m, PRO_MTP, EPI_STORE, s); }
    // App. B.2: the MTP head's decoder layer at the current latent position
    if (c->heads & PIPO_HEADS_MTP_LAYER) enqueue_layer(c, c->mtp, c->kc_mtp, c->vc_mtp, c->hd, c->ss_hd, s);
    // LM head #2 on RMSNorm(h_d; g_mo)
    GemvParams q{};
    q.B = B; q.eps = c->cfg.rms_eps; q.H = H; q.xh = c->xh; q.xl = c->xl; q.part = c->gpart; q.part_cap = c->gpart_cap;
    q.W = c->embed; q.N = c->V; q.K = H;
    q.x = c->hd; q.ss = c->ss_hd; q.nss = H / 16; q.gain = c->g_mtp_o;
    q.out = c->logits_d; q.best = c->best_d;
    { PROF_GEMV(PIPO_K_GEMV_LMHEAD); gemv(c, q, PRO_NORM, EPI_LOGITS, s); }
    if (!greedy) {
        // the draft's penalised set also holds its pair's backbone token
        PROF(PIPO_K_SAMPLE);
        launch_sample(sample_params(c, c->logits_d, B, 1, c->best_d, in_pair, c->best_b), s);
    }
    GateParams gp{};
    if (c->heads & PIPO_HEADS_MLP_CONFIDENCE) {
        // App. B.3: SiLU(W1 RMSNorm([h_b; h_d]; g_c)) into act; the gate takes w2 . act
        GemvParams f = gemv_base(c, B);
        f.W = c->conf_w1; f.N = H; f.K = 2 * H;
        f.x = c->x; f.x2 = c->hd; f.ss = c->ss_x; f.ss2 = c->ss_hd; f.nss = H / 16; f.gain = c->g_conf;
        f.act = c->act;
        { PROF_GEMV(PIPO_K_GEMV_SMALL); gemv(c, f, PRO_CAT, EPI_SILU, s); }
        gp.conf_h = c->act; gp.conf_w2 = c->conf_w2;
    }
    gp.hb = c->x; gp.hd = c->hd; gp.ss_b = c->ss_x; gp.nss_b = nss; gp.ss_d = c->ss_hd; gp.nss_d = H / 16;
    gp.w_conf = c->w_conf; gp.g_conf = c->g_conf; gp.H = H; gp.eps = c->cfg.rms_eps; gp.tau = c->tau;
    gp.best_b = c->best_b; gp.best_d = c->best_d; gp.pad_id = c->pad_id; gp.out = c->out;
    gp.pairs = c->pairs; gp.pos = c->pos; gp.step = c->step; gp.advance = advance; gp.B = B;
    if (c->eval_smp && in_pair) { gp.seen = c->seen; gp.seen_words = c->seen_words; gp.V = c->V; }
    PROF(PIPO_K_GATE);
    launch_gate(gp, s);
}

// One pair-decode step (eq. 1 on the pending pair, eq. 2 one position, heads).
static void enqueue_decode(pipo_ctx *c, hipStream_t s) {
    const int B = c->batch, H = c->H;
    if (c->heads & PIPO_HEADS_MLP_COMPRESSOR) {   // Table 4 MLP: E[a] + E[b] + W2 SiLU(W1 [E[a]; E[b]])
        GemvParams p = gemv_base(c, B);
        p.W = c->comp_w1; p.N = H; p.K = 2 * H; p.pairs = c->pairs; p.embed = c->embed; p.act = c->act;
        { PROF_GEMV(PIPO_K_GEMV_SMALL); gemv(c, p, PRO_PAIR, EPI_SILU, s); }
        { PROF(PIPO_K_GATE); launch_embed_step(c->pairs, c->embed, H, c->V, c->x, c->ss_x, B, 1, s); }
        p = gemv_base(c, B);
        p.W = c->comp_w2; p.N = H; p.K = H; p.xf = c->act; p.out = c->x; p.ss_out = c->ss_x;
        { PROF_GEMV(PIPO_K_GEMV_SMALL); gemv(c, p, PRO_F32, EPI_RESID, s); }
    } else {   // pair-in compressor, Linear (eq. 1)
        GemvParams p = gemv_base(c, B);
        p.W = c->w_comp; p.N = H; p.K = 2 * H; p.pairs = c->pairs; p.embed = c->embed;
        p.out = c->x; p.bias = c->b_comp; p.ss_out = c->ss_x;
        PROF_GEMV(PIPO_K_GEMV_SMALL);
        gemv(c, p, PRO_PAIR, EPI_STORE, s);
    }
    enqueue_layers(c, s);
    enqueue_heads(c, B, H / 16, 1, true, s);
}

static int check_sampling(pipo_ctx *c, const pipo_sampling *smp, int batch) {
    if (!smp) return fail(c, PIPO_EINVAL, "sampling is NULL");
    if (!(smp->tau == smp->tau)) return fail(c, PIPO_EINVAL, "tau is NaN");
    if (smp->temperature > 0.f) {
        if (!(smp->top_p > 0.f && smp->top_p <= 1.f)) return fail(c, PIPO_EINVAL, "top_p must be in (0, 1]");
        if (!smp->seeds) return fail(c, PIPO_EINVAL, "sampling needs per-sequence seeds");
        if (smp->top_k < 0) return fail(c, PIPO_EINVAL, "top_k must be >= 0");
        if (!(smp->rep_penalty > 0.f)) return fail(c, PIPO_EINVAL, "rep_penalty must be > 0");
    } else if (smp->top_k != 0 || smp->rep_penalty != 1.f) {
        return fail(c, PIPO_EINVAL, "top_k and rep_penalty apply to sampling (temperature > 0) only");
    }
    (void)batch;
    return PIPO_OK;
}

static int copy_outputs(pipo_ctx *c, pipo_pair *d_out, float *d_lb, float *d_ld, hipStream_t s) {
    const int B = c->batch;
    HIP_TRY(c, hipMemcpyAsync(d_out, c->out, sizeof(pipo_pair) * B, hipMemcpyDeviceToDevice, s));
    if (d_lb) HIP_TRY(c, hipMemcpyAsync(d_lb, c->logits_b, sizeof(float) * B * c->V, hipMemcpyDeviceToDevice, s));
    if (d_ld) HIP_TRY(c, hipMemcpyAsync(d_ld, c->logits_d, sizeof(float) * B * c->V, hipMemcpyDeviceToDevice, s));
    return PIPO_OK;
}

// The prompt prefill shared by both decoders: validation, sampling state,
// the chunked backbone over `positions` (PIPO: ceil(n/2) latents of
// compressed pairs, eq. 1; regular: the n tokens themselves), and the last
// position's residual into x.
// `n` is the row stride of d_tokens; `lens` (host [batch], or NULL: n each)
// the prompt lengths of a ragged batch.
static int prefill_backbone(pipo_ctx *c, int32_t batch, const int32_t *d_tokens, int32_t n, const int32_t *lens,
                            const pipo_sampling *smp, bool regular, hipStream_t s) {
    if (!d_tokens) return fail(c, PIPO_EINVAL, "d_tokens must be non-NULL");
    if (n < 1) return fail(c, PIPO_EINVAL, "prompt length must be >= 1 (got %d)", n);
    if (batch < 1) return fail(c, PIPO_EINVAL, "batch must be >= 1 (got %d)", batch);
    int rc = check_sampling(c, smp, batch);
    if (rc) return rc;
    if (batch > c->Bmax) return fail(c, PIPO_ECAPACITY, "batch %d exceeds max_batch %d", batch, c->Bmax);
    int nmax = n;
    if (lens) {
        nmax = 0;
        for (int b = 0; b < batch; ++b) {
            if (lens[b] < 1 || lens[b] > n)
                return fail(c, PIPO_EINVAL, "lens[%d] = %d outside [1, %d]", b, lens[b], n);
            nmax = std::max(nmax, (int)lens[b]);
        }
    }
    const int positions = regular ? nmax : (nmax + 1) / 2;   // the longest sequence's
    if (positions + 1 > c->cfg.max_latent)
        return fail(c, PIPO_ECAPACITY, "%d positions leave no room for a step (max_latent %d)", positions,
                    c->cfg.max_latent);
    HIP_TRY(c, hipGetLastError());
    // every host-side check has passed: from here the previous sequences are gone
    c->prefilled = false;
    c->enq_rc = PIPO_OK;

    if (c->batch != batch || c->tau != smp->tau || c->temperature != smp->temperature || c->top_p != smp->top_p ||
        c->top_k != smp->top_k || c->rep_penalty != smp->rep_penalty) {
        c->graph_dirty = true;
        c->graph_reg_dirty = true;
    }
    c->batch = batch;
    c->tau = smp->tau;
    c->temperature = smp->temperature;
    c->top_p = smp->top_p;
    c->top_k = smp->top_k;
    c->rep_penalty = smp->rep_penalty;
    c->eval_smp = smp->temperature > 0.f && (smp->top_k > 0 || smp->rep_penalty != 1.f);
    const int32_t *ntok = nullptr;
    if (lens) {
        HIP_TRY(c, hipEventSynchronize(c->lens_done));
        memcpy(c->h_lens, lens, sizeof(int32_t) * batch);
        HIP_TRY(c, hipMemcpyAsync(c->ntok, c->h_lens, sizeof(int32_t) * batch, hipMemcpyHostToDevice, s));
        HIP_TRY(c, hipEventRecord(c->lens_done, s));
        ntok = c->ntok;
    }
    if (c->eval_smp) {   // the prompt's tokens start each sequence's penalised set
        PROF(PIPO_K_PREFILL_MISC);
        launch_fill_u32(c->seen, 0u, (int64_t)batch * c->seen_words, s);
        launch_seen_mark(d_tokens, n, ntok, batch, c->V, c->seen, c->seen_words, s);
    }
    if (smp->temperature > 0.f) {
        HIP_TRY(c, hipEventSynchronize(c->seeds_done));
        memcpy(c->h_seeds, smp->seeds, sizeof(uint64_t) * batch);
        HIP_TRY(c, hipMemcpyAsync(c->seeds, c->h_seeds, sizeof(uint64_t) * batch, hipMemcpyHostToDevice, s));
        HIP_TRY(c, hipEventRecord(c->seeds_done, s));
    }
    const int H = c->H, F = c->F;
    PrefillGeom g{};
    for (int c0 = 0; c0 < positions; c0 += c->chunk) {
        g.B = batch; g.c0 = c0; g.clen = std::min(c->chunk, positions - c0);
        // ragged batches pad each sequence's rows to whole 64-row GEMM tiles, so
        // that tiles past a shorter prompt can be skipped
        g.mpad = (int)round_up(g.clen, ntok ? 64 : 32); g.n_tok = n; g.ntok = ntok; g.tok_per_pos = regular ? 1 : 2;
        const int M = batch * g.mpad;
        GemmParams gp{};
        gp.g = g; gp.M = M;
        gp.n_q = c->nq; gp.n_kv = c->nkv; gp.d = c->d; gp.lmax_pad = c->lmax_pad; gp.kv_bstride = c->kv_bstride;
        gp.rope_cos = c->rope_cos; gp.rope_sin = c->rope_sin;
        GemmParams p = gp;
        if (regular) {
            PROF(PIPO_K_PREFILL_MISC);
            launch_gather_tokens(d_tokens, c->embed, H, c->V, c->pad_id, g, c->p_x, s);
        } else if (c->heads & PIPO_HEADS_MLP_COMPRESSOR) {
            { PROF(PIPO_K_PREFILL_MISC); launch_gather_pairs(d_tokens, c->embed, H, c->V, c->pad_id, g, c->p_xin, s); }
            p.W = c->comp_w1; p.X = c->p_xin; p.N = H; p.K = 2 * H; p.epi = EPI_SILU; p.act_hi = c->p_act; p.act_lo = c->p_act_lo;
            { PROF(PIPO_K_PREFILL_GEMM); launch_gemm(p, s); }
            { PROF(PIPO_K_PREFILL_MISC); launch_gather_pair_sum(d_tokens, c->embed, H, c->V, c->pad_id, g, c->p_x, s); }
            p = gp;
            p.W = c->comp_w2; p.X = c->p_act; p.Xlo = c->p_act_lo; p.N = H; p.K = H; p.epi = EPI_RESID; p.out = c->p_x;
            { PROF(PIPO_K_PREFILL_GEMM); launch_gemm(p, s); }
        } else {
            { PROF(PIPO_K_PREFILL_MISC); launch_gather_pairs(d_tokens, c->embed, H, c->V, c->pad_id, g, c->p_xin, s); }
            p.W = c->w_comp; p.X = c->p_xin; p.N = H; p.K = 2 * H; p.epi = EPI_STORE; p.out = c->p_x; p.bias = c->b_comp;
            { PROF(PIPO_K_PREFILL_GEMM); launch_gemm(p, s); }
        }
        for (int l = 0; l < c->L; ++l) {
            const LayerW &lw = c->layers[l];
            uint16_t *kc = c->kc + (int64_t)l * c->Bmax * c->kv_bstride;
            uint16_t *vc = c->vc + (int64_t)l * c->Bmax * c->kv_bstride;
            { PROF(PIPO_K_PREFILL_MISC); launch_rmsnorm_tiled(c->p_x, lw.g_attn, H, c->cfg.rms_eps, M, c->p_xn, c->p_xn_lo, s); }
            p = gp;
            p.W = lw.wqkv; p.X = c->p_xn; p.Xlo = c->p_xn_lo; p.N = c->nqkv; p.K = H; p.epi = EPI_QKV; p.q = c->p_q; p.q_lo = c->p_q_lo; p.kc = kc; p.vc = vc;
            { PROF(PIPO_K_PREFILL_GEMM); launch_gemm(p, s); }
            AttnPrefillParams ap{};
            ap.q = c->p_q; ap.q_lo = c->p_q_lo; ap.kc = kc; ap.vc = vc; ap.kv_bstride = c->kv_bstride; ap.g = g;
            ap.n_q = c->nq; ap.n_kv = c->nkv; ap.d = c->d; ap.lmax_pad = c->lmax_pad; ap.out_hi = c->p_o; ap.out_lo = c->p_o_lo;
            { PROF(PIPO_K_PREFILL_ATTN); launch_attn_prefill(ap, s); }
            p = gp;
            p.W = lw.wo; p.X = c->p_o; p.Xlo = c->p_o_lo; p.N = H; p.K = c->qdim; p.epi = EPI_RESID; p.out = c->p_x;
            { PROF(PIPO_K_PREFILL_GEMM); launch_gemm(p, s); }
            { PROF(PIPO_K_PREFILL_MISC); launch_rmsnorm_tiled(c->p_x, lw.g_ffn, H, c->cfg.rms_eps, M, c->p_xn, c->p_xn_lo, s); }
            p = gp;
            p.W = lw.wgu; p.X = c->p_xn; p.Xlo = c->p_xn_lo; p.N = 2 * F; p.K = H; p.epi = EPI_SWIGLU; p.act_hi = c->p_act; p.act_lo = c->p_act_lo;
            { PROF(PIPO_K_PREFILL_GEMM); launch_gemm(p, s); }
            p = gp;
            p.W = lw.wdown; p.X = c->p_act; p.Xlo = c->p_act_lo; p.N = H; p.K = F; p.epi = EPI_RESID; p.out = c->p_x;
            { PROF(PIPO_K_PREFILL_GEMM); launch_gemm(p, s); }
        }
        // sequences whose last position is in this chunk take it as their step state
        { PROF(PIPO_K_PREFILL_MISC); launch_pick_last(c->p_x, H, g, c->x, c->ss_x, c->pos, c->step, regular, s); }
        if (!regular && (c->heads & PIPO_HEADS_MTP_LAYER)) {
            // App. B.2 over the chunk's latents (their K/V fill the MTP cache);
            // the MTP stream lives in p_xin, free once the compressor has run
            float *xm = (float *)c->p_xin;
            { PROF(PIPO_K_PREFILL_MISC);
              launch_mtp_rows(c->p_x, d_tokens, c->embed, c->g_mtp_h, c->g_mtp_e, H, c->V, c->pad_id, c->cfg.rms_eps, g, M,
                              c->p_act, c->p_act_lo, s); }
            p = gp;
            p.W = c->w_fc; p.X = c->p_act; p.Xlo = c->p_act_lo; p.N = H; p.K = 2 * H; p.epi = EPI_STORE; p.out = xm;
            { PROF(PIPO_K_PREFILL_GEMM); launch_gemm(p, s); }
            const LayerW &lw = c->mtp;
            { PROF(PIPO_K_PREFILL_MISC); launch_rmsnorm_tiled(xm, lw.g_attn, H, c->cfg.rms_eps, M, c->p_xn, c->p_xn_lo, s); }
            p = gp;
            p.W = lw.wqkv; p.X = c->p_xn; p.Xlo = c->p_xn_lo; p.N = c->nqkv; p.K = H; p.epi = EPI_QKV; p.q = c->p_q; p.q_lo = c->p_q_lo;
            p.kc = c->kc_mtp; p.vc = c->vc_mtp;
            { PROF(PIPO_K_PREFILL_GEMM); launch_gemm(p, s); }
            AttnPrefillParams ap{};
            ap.q = c->p_q; ap.q_lo = c->p_q_lo; ap.kc = c->kc_mtp; ap.vc = c->vc_mtp; ap.kv_bstride = c->kv_bstride; ap.g = g;
            ap.n_q = c->nq; ap.n_kv = c->nkv; ap.d = c->d; ap.lmax_pad = c->lmax_pad; ap.out_hi = c->p_o; ap.out_lo = c->p_o_lo;
            { PROF(PIPO_K_PREFILL_ATTN); launch_attn_prefill(ap, s); }
            p = gp;
            p.W = lw.wo; p.X = c->p_o; p.Xlo = c->p_o_lo; p.N = H; p.K = c->qdim; p.epi = EPI_RESID; p.out = xm;
            { PROF(PIPO_K_PREFILL_GEMM); launch_gemm(p, s); }
            { PROF(PIPO_K_PREFILL_MISC); launch_rmsnorm_tiled(xm, lw.g_ffn, H, c->cfg.rms_eps, M, c->p_xn, c->p_xn_lo, s); }
            p = gp;
            p.W = lw.wgu; p.X = c->p_xn; p.Xlo = c->p_xn_lo; p.N = 2 * F; p.K = H; p.epi = EPI_SWIGLU; p.act_hi = c->p_act; p.act_lo = c->p_act_lo;
            { PROF(PIPO_K_PREFILL_GEMM); launch_gemm(p, s); }
            p = gp;
            p.W = lw.wdown; p.X = c->p_act; p.Xlo = c->p_act_lo; p.N = H; p.K = F; p.epi = EPI_RESID; p.out = xm;
            { PROF(PIPO_K_PREFILL_GEMM); launch_gemm(p, s); }
        }
    }
    c->len = positions;
    return PIPO_OK;
}

static int prefill_pair(pipo_ctx *c, int32_t batch, const int32_t *d_tokens, int32_t n, const int32_t *lens,
                        const pipo_sampling *smp, pipo_pair *d_out, float *d_logits_b, float *d_logits_d,
                        void *stream) {
    if (!c) return fail(nullptr, PIPO_EINVAL, "ctx is NULL");
    if (!d_out) return fail(c, PIPO_EINVAL, "d_out must be non-NULL");
    hipStream_t s = (hipStream_t)stream;
    int rc = prefill_backbone(c, batch, d_tokens, n, lens, smp, false, s);
    if (rc) return rc;
    enqueue_heads(c, batch, c->H / 16, 1, false, s);
    HIP_TRY(c, hipGetLastError());
    if (c->enq_rc) return c->enq_rc;
    rc = copy_outputs(c, d_out, d_logits_b, d_logits_d, s);
    if (rc) return rc;
    c->prefilled = true;
    c->regular = false;
    return PIPO_OK;
}

extern "C" int pipo_prefill(pipo_ctx *c, int32_t batch, const int32_t *d_tokens, int32_t n,
                            const pipo_sampling *smp, pipo_pair *d_out, float *d_logits_b, float *d_logits_d,
                            void *stream) {
    return prefill_pair(c, batch, d_tokens, n, nullptr, smp, d_out, d_logits_b, d_logits_d, stream);
}

extern "C" int pipo_prefill_ragged(pipo_ctx *c, int32_t batch, const int32_t *d_tokens, int32_t stride,
                                   const int32_t *lens, const pipo_sampling *smp, pipo_pair *d_out,
                                   float *d_logits_b, float *d_logits_d, void *stream) {
    if (!lens) return fail(c, PIPO_EINVAL, "lens must be non-NULL");
    return prefill_pair(c, batch, d_tokens, stride, lens, smp, d_out, d_logits_b, d_logits_d, stream);
}

// Regular decoding's heads: eq. 3 alone (tied LM head on RMSNorm(h; g_final),
// greedy or top-p in sampler slot 0), then the token becomes the next input.
static void enqueue_regular_heads(pipo_ctx *c, int B, int nss, int advance, bool in_tok, hipStream_t s) {
    const bool greedy = c->temperature <= 0.f;
    GemvParams p{};
    p.B = B; p.eps = c->cfg.rms_eps; p.H = c->H; p.xh = c->xh; p.xl = c->xl; p.part = c->gpart; p.part_cap = c->gpart_cap;
    p.W = c->embed; p.N = c->V; p.K = c->H;
    p.x = c->x; p.ss = c->ss_x; p.nss = nss; p.gain = c->g_final;
    p.out = c->logits_b; p.best = c->best_b;   // sampling reads the row max from the key
    { PROF_GEMV(PIPO_K_GEMV_LMHEAD); gemv(c, p, PRO_NORM, EPI_LOGITS, s); }
    if (!greedy) {
        PROF(PIPO_K_SAMPLE);
        launch_sample(sample_params(c, c->logits_b, B, 0, c->best_b, in_tok, nullptr), s);
    }
    PROF(PIPO_K_GATE);
    const bool mark = c->eval_smp && in_tok;   // the step's input token joins the penalised set
    launch_regular_out(c->best_b, c->out_tok, c->pairs, c->pad_id, c->pos, c->step, advance, B,
                       mark ? c->seen : nullptr, c->seen_words, c->V, s);
}

// One regular decoding step: x = E[token] at the next position, the same
// backbone layers as the pair step (eq. 2 for one position), the heads above.
static void enqueue_regular_decode(pipo_ctx *c, hipStream_t s) {
    const int B = c->batch, H = c->H;
    { PROF(PIPO_K_GATE); launch_embed_step(c->pairs, c->embed, H, c->V, c->x, c->ss_x, B, 0, s); }
    enqueue_layers(c, s);
    enqueue_regular_heads(c, B, H / 16, 1, true, s);
}

static int copy_tokens(pipo_ctx *c, int32_t *d_tok, float *d_logits, hipStream_t s) {
    const int B = c->batch;
    HIP_TRY(c, hipMemcpyAsync(d_tok, c->out_tok, sizeof(int32_t) * B, hipMemcpyDeviceToDevice, s));
    if (d_logits) HIP_TRY(c, hipMemcpyAsync(d_logits, c->logits_b, sizeof(float) * B * c->V, hipMemcpyDeviceToDevice, s));
    return PIPO_OK;
}

static int prefill_regular(pipo_ctx *c, int32_t batch, const int32_t *d_tokens, int32_t n, const int32_t *lens,
                           const pipo_sampling *smp, int32_t *d_tok, float *d_logits, void *stream) {
    if (!c) return fail(nullptr, PIPO_EINVAL, "ctx is NULL");
    if (!d_tok) return fail(c, PIPO_EINVAL, "d_tok must be non-NULL");
    hipStream_t s = (hipStream_t)stream;
    int rc = prefill_backbone(c, batch, d_tokens, n, lens, smp, true, s);
    if (rc) return rc;
    enqueue_regular_heads(c, batch, c->H / 16, 1, false, s);
    HIP_TRY(c, hipGetLastError());
    if (c->enq_rc) return c->enq_rc;
    rc = copy_tokens(c, d_tok, d_logits, s);
    if (rc) return rc;
    c->prefilled = true;
    c->regular = true;
    return PIPO_OK;
}

extern "C" int pipo_regular_prefill(pipo_ctx *c, int32_t batch, const int32_t *d_tokens, int32_t n,
                                    const pipo_sampling *smp, int32_t *d_tok, float *d_logits, void *stream) {
    return prefill_regular(c, batch, d_tokens, n, nullptr, smp, d_tok, d_logits, stream);
}

extern "C" int pipo_regular_prefill_ragged(pipo_ctx *c, int32_t batch, const int32_t *d_tokens, int32_t stride,
                                           const int32_t *lens, const pipo_sampling *smp, int32_t *d_tok,
                                           float *d_logits, void *stream) {
    if (!lens) return fail(c, PIPO_EINVAL, "lens must be non-NULL");
    return prefill_regular(c, batch, d_tokens, stride, lens, smp, d_tok, d_logits, stream);
}

extern "C" int pipo_regular_step(pipo_ctx *c, const int32_t *d_in_tok, int32_t *d_tok, float *d_logits,
                                 void *stream) {
    if (!c) return fail(nullptr, PIPO_EINVAL, "ctx is NULL");
    if (!d_tok) return fail(c, PIPO_EINVAL, "d_tok must be non-NULL");
    if (!c->prefilled || !c->regular) return fail(c, PIPO_ESTATE, "regular step before a regular prefill");
    if (c->len + 1 > c->cfg.max_latent)
        return fail(c, PIPO_ECAPACITY, "KV cache full: %d positions, max_latent %d", c->len, c->cfg.max_latent);
    hipStream_t s = (hipStream_t)stream;
    HIP_TRY(c, hipGetLastError());
    if (d_in_tok)   // teacher forcing: the input tokens into the first slot of each pair
        HIP_TRY(c, hipMemcpy2DAsync(c->pairs, 2 * sizeof(int32_t), d_in_tok, sizeof(int32_t), sizeof(int32_t),
                                    c->batch, hipMemcpyDeviceToDevice, s));
    if (c->use_graph && !c->prof_on) {
        if (c->graph_reg_dirty || !c->graph_reg) {
            if (c->graph_reg) {
                hipGraphExecDestroy(c->graph_reg);
                c->graph_reg = nullptr;
            }
            hipGraph_t gr;
            c->enq_rc = PIPO_OK;
            HIP_TRY(c, hipStreamBeginCapture(c->cap_stream, hipStreamCaptureModeThreadLocal));
            enqueue_regular_decode(c, c->cap_stream);
            HIP_TRY(c, hipStreamEndCapture(c->cap_stream, &gr));
            if (c->enq_rc) {
                hipGraphDestroy(gr);
                return c->enq_rc;
            }
            hipError_t e = hipGraphInstantiate(&c->graph_reg, gr, nullptr, nullptr, 0);
            hipGraphDestroy(gr);
            if (e != hipSuccess) return fail(c, PIPO_EHIP, "graph instantiate: %s", hipGetErrorString(e));
            c->graph_reg_dirty = false;
        }
        HIP_TRY(c, hipGraphLaunch(c->graph_reg, s));
    } else {
        c->enq_rc = PIPO_OK;
        enqueue_regular_decode(c, s);
        HIP_TRY(c, hipGetLastError());
        if (c->enq_rc) return c->enq_rc;
    }
    int rc = copy_tokens(c, d_tok, d_logits, s);
    if (rc) return rc;
    c->len += 1;
    return PIPO_OK;
}

extern "C" int pipo_decode_step(pipo_ctx *c, const int32_t *d_in_pairs, pipo_pair *d_out, float *d_logits_b,
                                float *d_logits_d, void *stream) {
    if (!c) return fail(nullptr, PIPO_EINVAL, "ctx is NULL");
    if (!d_out) return fail(c, PIPO_EINVAL, "d_out must be non-NULL");
    if (!c->prefilled || c->regular) return fail(c, PIPO_ESTATE, "decode step before a PIPO prefill");
    if (c->len + 1 > c->cfg.max_latent)
        return fail(c, PIPO_ECAPACITY, "KV cache full: %d latents, max_latent %d", c->len, c->cfg.max_latent);
    hipStream_t s = (hipStream_t)stream;
    HIP_TRY(c, hipGetLastError());
    if (d_in_pairs)
        HIP_TRY(c, hipMemcpyAsync(c->pairs, d_in_pairs, sizeof(int32_t) * 2 * c->batch, hipMemcpyDeviceToDevice, s));
    if (c->use_graph && !c->prof_on) {
        if (c->graph_dirty || !c->graph) {
            if (c->graph) {
                hipGraphExecDestroy(c->graph);
                c->graph = nullptr;
            }
            hipGraph_t gr;
            c->enq_rc = PIPO_OK;
            HIP_TRY(c, hipStreamBeginCapture(c->cap_stream, hipStreamCaptureModeThreadLocal));
            enqueue_decode(c, c->cap_stream);
            HIP_TRY(c, hipStreamEndCapture(c->cap_stream, &gr));
            if (c->enq_rc) {
                hipGraphDestroy(gr);
                return c->enq_rc;
            }
            hipError_t e = hipGraphInstantiate(&c->graph, gr, nullptr, nullptr, 0);
            hipGraphDestroy(gr);
            if (e != hipSuccess) return fail(c, PIPO_EHIP, "graph instantiate: %s", hipGetErrorString(e));
            c->graph_dirty = false;
        }
        HIP_TRY(c, hipGraphLaunch(c->graph, s));
    } else {
        c->enq_rc = PIPO_OK;
        enqueue_decode(c, s);
        HIP_TRY(c, hipGetLastError());
        if (c->enq_rc) return c->enq_rc;
    }
    int rc = copy_outputs(c, d_out, d_logits_b, d_logits_d, s);
    if (rc) return rc;
    c->len += 1;
    return PIPO_OK;
}

// The pair step of pipo_decode_step, launched eagerly on the caller's stream
// with the attention and k-range partials in the device's static scratch:
// no allocation and no graph instantiation, so a caller under HIP graph
// capture can record it.
extern "C" int pipo_decode_step_noalloc(pipo_ctx *c, const int32_t *d_in_pairs, pipo_pair *d_out,
                                        float *d_logits_b, float *d_logits_d, void *stream) {
    if (!c) return fail(nullptr, PIPO_EINVAL, "ctx is NULL");
    if (!d_out) return fail(c, PIPO_EINVAL, "d_out must be non-NULL");
    if (!c->prefilled || c->regular) return fail(c, PIPO_ESTATE, "decode step before a PIPO prefill");
    if (c->len + 1 > c->cfg.max_latent)
        return fail(c, PIPO_ECAPACITY, "KV cache full: %d latents, max_latent %d", c->len, c->cfg.max_latent);
    if (!c->scratch) return fail(c, PIPO_EHIP, "no scratch address for device %d", c->dev);
    const int64_t attn_floats =
        round_up((int64_t)c->batch * c->nq * attn_splits(c, c->batch) * attn_part_stride(c->d), 64);
    const int64_t cap_floats = (int64_t)(kScratchBytes / sizeof(float));
    if (attn_floats > cap_floats)
        return fail(c, PIPO_ECAPACITY, "attention partials of %lld bytes exceed the %zu-byte scratch",
                    (long long)(attn_floats * 4), kScratchBytes);
    hipStream_t s = (hipStream_t)stream;
    HIP_TRY(c, hipGetLastError());
    if (d_in_pairs)
        HIP_TRY(c, hipMemcpyAsync(c->pairs, d_in_pairs, sizeof(int32_t) * 2 * c->batch, hipMemcpyDeviceToDevice, s));
    // this call's partials live in the scratch; the GEMVs whose k-range
    // partials do not fit the rest take their whole-K path instead
    float *const apart = c->apart, *const gpart = c->gpart;
    const int64_t gcap = c->gpart_cap;
    const bool prof = c->prof_on;
    c->apart = (float *)c->scratch;
    c->gpart = c->apart + attn_floats;
    c->gpart_cap = cap_floats - attn_floats;
    c->prof_on = false;   // no events: profiling does not cover this call
    c->enq_rc = PIPO_OK;
    enqueue_decode(c, s);
    c->apart = apart;
    c->gpart = gpart;
    c->gpart_cap = gcap;
    c->prof_on = prof;
    HIP_TRY(c, hipGetLastError());
    if (c->enq_rc) return c->enq_rc;
    int rc = copy_outputs(c, d_out, d_logits_b, d_logits_d, s);
    if (rc) return rc;
    c->len += 1;
    return PIPO_OK;
}

extern "C" int pipo_profile_enable(pipo_ctx *c, int on) {
    if (!c) return fail(nullptr, PIPO_EINVAL, "ctx is NULL");
    c->prof_on = on != 0;
    c->pending.clear();
    c->ev_next = 0;
    for (int k = 0; k < PIPO_K_CLASSES; ++k) { c->prof_ms[k] = 0.0; c->prof_n[k] = 0; }
    return PIPO_OK;
}

extern "C" int pipo_profile_read(pipo_ctx *c, int kclass, double *total_ms, int64_t *launches) {
    if (!c) return fail(nullptr, PIPO_EINVAL, "ctx is NULL");
    if (kclass < 0 || kclass >= PIPO_K_CLASSES || !total_ms || !launches)
        return fail(c, PIPO_EINVAL, "bad profiling arguments");
    for (auto &pr : c->pending) {
        HIP_TRY(c, hipEventSynchronize(c->ev_pool[pr.second + 1]));
        float ms = 0.f;
        HIP_TRY(c, hipEventElapsedTime(&ms, c->ev_pool[pr.second], c->ev_pool[pr.second + 1]));
        c->prof_ms[pr.first] += ms;
        c->prof_n[pr.first] += 1;
    }
    c->pending.clear();
    c->ev_next = 0;
    *total_ms = c->prof_ms[kclass];
    *launches = c->prof_n[kclass];
    return PIPO_OK;
}

extern "C" int pipo_free(pipo_ctx *c) {
    if (!c) return PIPO_OK;
    for (hipEvent_t e : c->ev_pool) hipEventDestroy(e);
    if (c->graph) hipGraphExecDestroy(c->graph);
    if (c->graph_reg) hipGraphExecDestroy(c->graph_reg);
    if (c->cap_stream) hipStreamDestroy(c->cap_stream);
    if (c->seeds_done) hipEventDestroy(c->seeds_done);
    if (c->h_seeds) hipHostFree(c->h_seeds);
    if (c->lens_done) hipEventDestroy(c->lens_done);
    if (c->h_lens) hipHostFree(c->h_lens);
    if (c->wmem) hipFree(c->wmem);
    if (c->amem) hipFree(c->amem);
    delete c;
    return PIPO_OK;
}

extern "C" const char *pipo_last_error(const pipo_ctx *c) {
    return c ? c->err.c_str() : g_init_error.c_str();
}

extern "C" int pipo_read_weight(pipo_ctx *c, const char *name, int64_t start, int64_t count, uint16_t *host_out) {
    if (!c) return fail(nullptr, PIPO_EINVAL, "ctx is NULL");
    if (!name || !host_out || start < 0 || count < 0) return fail(c, PIPO_EINVAL, "bad arguments");
    const int H = c->H, F = c->F;
    const uint16_t *src = nullptr;
    const float *vec = nullptr;
    int64_t N = 0, K = 0, row_base = 0, rows_total = 0, off = 0;
    int perm = PERM_NONE, half = 0;
    std::string nm(name);
    int layer = -1;
    if (nm.rfind("mtp.", 0) == 0) {
        if (!(c->heads & PIPO_HEADS_MTP_LAYER)) return fail(c, PIPO_EINVAL, "no MTP layer in this model: %s", name);
        layer = c->L;   // the MTP head's decoder layer
        nm = nm.substr(4);
    } else if (nm.size() > 1 && nm[0] == 'l' && nm.find('.') != std::string::npos) {
        layer = atoi(nm.c_str() + 1);
        if (layer < 0 || layer >= c->L) return fail(c, PIPO_EINVAL, "layer out of range in %s", name);
        nm = nm.substr(nm.find('.') + 1);
    }
    if (layer < 0) {
        if (nm == "embed") { src = c->embed; N = c->V; K = H; }
        else if (nm == "w_comp") { src = c->w_comp; N = H; K = 2 * H; }
        else if (nm == "w_fc") { src = c->w_fc; N = H; K = 2 * H; }
        else if (nm == "b_comp") { vec = c->b_comp; N = H; }
        else if (nm == "w_conf") { vec = c->w_conf; N = 2 * H; }
        else if (nm == "g_final") { vec = c->g_final; N = H; }
        else if (nm == "g_mtp_h") { vec = c->g_mtp_h; N = H; }
        else if (nm == "g_mtp_e") { vec = c->g_mtp_e; N = H; }
        else if (nm == "g_mtp_o") { vec = c->g_mtp_o; N = H; }
        else if (nm == "g_conf") { vec = c->g_conf; N = 2 * H; }
        else if (nm == "comp_w1" && c->comp_w1) { src = c->comp_w1; N = H; K = 2 * H; }
        else if (nm == "comp_w2" && c->comp_w2) { src = c->comp_w2; N = H; K = H; }
        else if (nm == "conf_w1" && c->conf_w1) { src = c->conf_w1; N = H; K = 2 * H; }
        else if (nm == "conf_w2" && c->conf_w2) { vec = c->conf_w2; N = H; }
    } else {
        const LayerW &lw = layer < c->L ? c->layers[layer] : c->mtp;
        if (nm == "wq") { src = lw.wqkv; N = c->qdim; K = H; perm = PERM_QK; half = c->d / 2; }
        else if (nm == "wk") { src = lw.wqkv; N = c->kvdim; K = H; perm = PERM_QK; half = c->d / 2; row_base = c->qdim; }
        else if (nm == "wv") { src = lw.wqkv; N = c->kvdim; K = H; row_base = c->qdim + c->kvdim; }
        else if (nm == "wo") { src = lw.wo; N = H; K = c->qdim; }
        else if (nm == "wgate") { src = lw.wgu; N = F; K = H; perm = PERM_GATEUP; rows_total = F; }
        else if (nm == "wup") { src = lw.wgu; N = F; K = H; perm = PERM_GATEUP; rows_total = F; off = (int64_t)F * H; }
        else if (nm == "wdown") { src = lw.wdown; N = H; K = F; }
        else if (nm == "g_attn") { vec = lw.g_attn; N = H; }
        else if (nm == "g_ffn") { vec = lw.g_ffn; N = H; }
    }
    if (!src && !vec) return fail(c, PIPO_EINVAL, "unknown tensor %s", name);
    const int64_t total = vec ? N : N * K;
    if (start + count > total) return fail(c, PIPO_EINVAL, "range past the end of %s", name);
    if (count == 0) return PIPO_OK;
    if (vec) {
        std::vector<float> tmp(count);
        HIP_TRY(c, hipMemcpy(tmp.data(), vec + start, sizeof(float) * count, hipMemcpyDeviceToHost));
        for (int64_t i = 0; i < count; ++i) {
            uint32_t u;
            memcpy(&u, &tmp[i], 4);
            host_out[i] = (uint16_t)(u >> 16);   // values are bf16-exact
        }
        return PIPO_OK;
    }
    uint16_t *dtmp = nullptr;
    HIP_TRY(c, hipMalloc(&dtmp, sizeof(uint16_t) * count));
    launch_read_tiled(src, N, K, start + off, count, perm, half, row_base, rows_total, dtmp, nullptr);
    hipError_t e = hipMemcpy(host_out, dtmp, sizeof(uint16_t) * count, hipMemcpyDeviceToHost);
    hipFree(dtmp);
    if (e != hipSuccess) return fail(c, PIPO_EHIP, "read back: %s", hipGetErrorString(e));
    return PIPO_OK;
}
