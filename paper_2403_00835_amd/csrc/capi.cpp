// Runtime of libcllm.so: device memory, weight repacking, the iteration launch sequence, the
// device-resident decode loop and the C ABI of include/cllm.h.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "../../include/cllm.h"
#include "device.h"
#include "launch.h"

using namespace cllm;

struct cllm_ctx {
    cllm_config cfg{};
    cllm_runtime_opts opts{};
    hipStream_t stream = nullptr;
    bool bf16 = true;
    int elem = 2;
    int d = 0, H = 0, hd = 0, F = 0, V = 0, NL = 0;
    int Fp = 0;         // ffn width padded to 32
    int ctx_alloc = 0;  // KV capacity, multiple of the attention chunk
    int nch = 0;        // attention chunks of ctx_alloc
    int ks_d = 0, ks_f = 0;
    int n_wg_qkv = 0, n_wg_o = 0, n_wg_gu = 0, n_wg_d = 0, n_wg_lm = 0;
    int64_t streamed_bytes = 0;

    // weights
    void *embed = nullptr;
    std::vector<float *> g_attn, g_ffn;
    float *g_final = nullptr;
    std::vector<uint8_t *> w_qkv, w_o, w_gu, w_d;
    uint8_t *w_lm = nullptr;
    // KV cache: K [layer][ctx_alloc][d], V transposed [layer][d][ctx_alloc]
    void *kc = nullptr, *vt = nullptr;
    float *rcos = nullptr, *rsin = nullptr;
    // workspace
    float *X = nullptr, *ssq = nullptr, *pmax = nullptr, *opart = nullptr, *mpart = nullptr, *lpart = nullptr,
          *dbg = nullptr;
    int *pidx = nullptr;
    void *Q = nullptr, *O = nullptr, *Hb = nullptr;
    void *An = nullptr;  // RMSNorm operand x (.) g of the next normed product
    Ctl *ctl = nullptr;
    int32_t *out_dev = nullptr, *stream_dev = nullptr;
    int stream_cap = 0;
    std::vector<void *> allocs;

    // host state
    bool prefilled = false;
    int L = 0, pending = 0;
    bool dead = false;
    std::string err;
    bool dbg_on = false;
    float *dbg_host = nullptr;
    size_t dbg_cap = 0;
    // kernel timing
    int kt_class = -1;
    int kt_rg = 0;  // time only launches for this many 16-row groups (0 = all)
    std::vector<hipEvent_t> ev_pool;
    size_t ev_used = 0;
    int64_t kt_launches = 0;
    double kt_ms = 0.0;
};

namespace {

cllm_status fail(cllm_ctx *c, cllm_status s, const char *fmt, ...) {
    if (c) {
        char buf[512];
        va_list ap;
        va_start(ap, fmt);
        vsnprintf(buf, sizeof buf, fmt, ap);
        va_end(ap);
        c->err = buf;
        if (s == CLLM_ERR_DEVICE) c->dead = true;
    }
    return s;
}

#define HIPCHK(c, expr)                                                                            \
    do {                                                                                           \
        hipError_t _e = (expr);                                                                    \
        if (_e != hipSuccess)                                                                      \
            return fail((c), CLLM_ERR_DEVICE, "%s failed: %s (%s:%d)", #expr, hipGetErrorString(_e), \
                        __FILE__, __LINE__);                                                       \
    } while (0)

inline int round_up(int x, int a) { return (x + a - 1) / a * a; }
inline int rows_to_rg(int rows) { return rows <= 16 ? 1 : (rows <= 32 ? 2 : 4); }

cllm_status dalloc(cllm_ctx *c, void **p, size_t bytes) {
    if (bytes == 0) bytes = 16;
    hipError_t e = hipMalloc(p, bytes);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        *p = nullptr;
        return fail(c, CLLM_ERR_OOM, "hipMalloc(%zu) failed: %s", bytes, hipGetErrorString(e));
    }
    c->allocs.push_back(*p);
    e = hipMemsetAsync(*p, 0, bytes, c->stream);
    if (e != hipSuccess) return fail(c, CLLM_ERR_DEVICE, "hipMemsetAsync failed: %s", hipGetErrorString(e));
    return CLLM_OK;
}

template <class T>
cllm_status dalloc_t(cllm_ctx *c, T **p, size_t count) {
    void *v = nullptr;
    cllm_status s = dalloc(c, &v, count * sizeof(T));
    *p = reinterpret_cast<T *>(v);
    return s;
}

// Timing events for the selected kernel class and row-group count (null when not timed).
void timing_events(cllm_ctx *c, int cls, int rg, hipEvent_t *e0, hipEvent_t *e1) {
    *e0 = *e1 = nullptr;
    if (c->kt_class != cls || (c->kt_rg > 0 && c->kt_rg != rg)) return;
    while (c->ev_pool.size() < c->ev_used + 2) {
        hipEvent_t e;
        if (hipEventCreate(&e) != hipSuccess) return;
        c->ev_pool.push_back(e);
    }
    *e0 = c->ev_pool[c->ev_used];
    *e1 = c->ev_pool[c->ev_used + 1];
    c->ev_used += 2;
}

void timing_collect(cllm_ctx *c) {
    for (size_t i = 0; i + 1 < c->ev_used; i += 2) {
        float ms = 0.f;
        if (hipEventElapsedTime(&ms, c->ev_pool[i], c->ev_pool[i + 1]) == hipSuccess) {
            c->kt_ms += ms;
            c->kt_launches += 1;
        }
    }
    c->ev_used = 0;
}

// Host-side row order of a packed GEMM (the logical source row of each packed row, -1 = zero).
std::vector<int32_t> qkv_perm(const cllm_ctx *c) {
    const int d = c->d, hd = c->hd, h2 = hd / 2;
    std::vector<int32_t> p(3 * d);
    for (int R = 0; R < 3 * d; ++R) {
        const int sec = R / d, within = R % d, head = within / hd, q = within % hd;
        int dim = q;
        if (hd >= 32) {
            const int b16 = q >> 4, o = q & 15;
            dim = (b16 & 1) ? (h2 + (b16 >> 1) * 16 + o) : ((b16 >> 1) * 16 + o);
        }
        p[R] = sec * d + head * hd + dim;
    }
    return p;
}

std::vector<int32_t> gate_up_perm(const cllm_ctx *c) {
    std::vector<int32_t> p(2 * c->Fp);
    for (int R = 0; R < 2 * c->Fp; ++R) {
        const int t = R / 16, o = R % 16, f = (t / 2) * 16 + o;
        p[R] = f < c->F ? ((t & 1) ? c->F + f : f) : -1;
    }
    return p;
}

std::vector<int32_t> plain_perm(int rows_padded, int rows) {
    std::vector<int32_t> p(rows_padded);
    for (int r = 0; r < rows_padded; ++r) p[r] = r < rows ? r : -1;
    return p;
}

// Upload one logical [N][K] matrix (host) and repack it into tiles.
// Ks is the k-step count of the packed layout (K rounded up; the padding is zero).
cllm_status upload_packed(cllm_ctx *c, const void *host, int N, int K, int Ks, const std::vector<int32_t> &perm,
                          uint8_t **dst, void *staging, int32_t *perm_dev) {
    const int n_tiles = (int)perm.size() / 16;
    const size_t bytes = (size_t)n_tiles * Ks * kTileBytes;
    if (!*dst) {
        cllm_status s = dalloc(c, reinterpret_cast<void **>(dst), bytes);
        if (s) return s;
    }
    HIPCHK(c, hipMemcpyAsync(staging, host, (size_t)N * K * c->elem, hipMemcpyHostToDevice, c->stream));
    HIPCHK(c, hipMemcpyAsync(perm_dev, perm.data(), perm.size() * sizeof(int32_t), hipMemcpyHostToDevice, c->stream));
    HIPCHK(c, launch_repack(c->bf16, staging, perm_dev, K, Ks, n_tiles, *dst, c->stream));
    HIPCHK(c, hipStreamSynchronize(c->stream));  // staging and perm are reused
    c->streamed_bytes += (int64_t)bytes;
    return CLLM_OK;
}

// One iteration's launch sequence for up to `rows` rows (the device control block holds m).
cllm_status enqueue_iteration(cllm_ctx *c, int rows, int nch_launch, bool with_lm, int32_t *out_dev,
                              const int32_t *stream_dev) {
    const int rg = rows_to_rg(rows);
    hipStream_t s = c->stream;
    hipEvent_t e0, e1;

    EmbedParams ep{c->embed, c->X, c->ssq, c->An, c->g_attn[0], c->d, c->ctl};
    timing_events(c, CLLM_KT_EMBED, rg, &e0, &e1);
    HIPCHK(c, launch_embed(c->bf16, 16 * rg, ep, s, e0, e1));

    GemmParams base{};
    base.ctl = c->ctl;
    base.ssq = c->ssq;
    base.T = c->d / 16;
    base.K = c->d;
    base.eps = c->cfg.rms_eps;
    base.d = c->d;
    base.hd = c->hd;
    base.ctx_alloc = c->ctx_alloc;
    base.rcos = c->rcos;
    base.rsin = c->rsin;
    base.Xout = c->X;
    base.ssq_out = c->ssq;
    base.ldx = c->d;
    base.An = c->An;
    base.Fp = c->Fp;
    base.V = c->V;

    AttnParams ap{};
    ap.Q = c->Q;
    ap.O = c->O;
    ap.Opart = c->opart;
    ap.Mpart = c->mpart;
    ap.Lpart = c->lpart;
    ap.d = c->d;
    ap.hd = c->hd;
    ap.n_heads = c->H;
    ap.nch = c->nch;
    ap.ctx_alloc = c->ctx_alloc;
    ap.scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)c->hd));
    ap.ctl = c->ctl;

    const size_t kv_layer = (size_t)c->ctx_alloc * c->d * c->elem;
    for (int l = 0; l < c->NL; ++l) {
        void *kc = static_cast<uint8_t *>(c->kc) + l * kv_layer;
        void *vt = static_cast<uint8_t *>(c->vt) + l * kv_layer;

        GemmParams q = base;  // operand: attention RMSNorm of X, written by the previous producer
        q.W = c->w_qkv[l];
        q.Ks = c->ks_d;
        q.n_wg = c->n_wg_qkv;
        q.A = c->An;
        q.lda = c->d;
        q.Q = c->Q;
        q.Kc = kc;
        q.Vt = vt;
        timing_events(c, CLLM_KT_GEMM_QKV, rg, &e0, &e1);
        HIPCHK(c, launch_gemm(GEMM_QKV, c->bf16, rg, q, s, e0, e1));

        ap.Kc = kc;
        ap.Vt = vt;
        timing_events(c, CLLM_KT_ATTN, rg, &e0, &e1);
        HIPCHK(c, launch_attn(c->bf16, rg, nch_launch, ap, s, e0, e1));
        timing_events(c, CLLM_KT_ATTN_COMBINE, rg, &e0, &e1);
        HIPCHK(c, launch_attn_combine(c->bf16, 16 * rg, ap, s, e0, e1));

        GemmParams o = base;  // X += O W_o^T; writes the FFN RMSNorm operand
        o.W = c->w_o[l];
        o.Ks = c->ks_d;
        o.n_wg = c->n_wg_o;
        o.A = c->O;
        o.lda = c->d;
        o.gain = c->g_ffn[l];
        timing_events(c, CLLM_KT_GEMM_O, rg, &e0, &e1);
        HIPCHK(c, launch_gemm(GEMM_O, c->bf16, rg, o, s, e0, e1));

        GemmParams gu = base;
        gu.W = c->w_gu[l];
        gu.Ks = c->ks_d;
        gu.n_wg = c->n_wg_gu;
        gu.A = c->An;
        gu.lda = c->d;
        gu.H = c->Hb;
        timing_events(c, CLLM_KT_GEMM_GATE_UP, rg, &e0, &e1);
        HIPCHK(c, launch_gemm(GEMM_GATE_UP, c->bf16, rg, gu, s, e0, e1));

        GemmParams dn = base;  // X += H W_d^T; writes the next layer's (or the final) RMSNorm operand
        dn.W = c->w_d[l];
        dn.Ks = c->ks_f;
        dn.n_wg = c->n_wg_d;
        dn.A = c->Hb;
        dn.lda = c->Fp;
        dn.gain = l + 1 < c->NL ? c->g_attn[l + 1] : c->g_final;
        timing_events(c, CLLM_KT_GEMM_DOWN, rg, &e0, &e1);
        HIPCHK(c, launch_gemm(GEMM_DOWN, c->bf16, rg, dn, s, e0, e1));
    }

    ScanParams sp{};
    sp.ctl = c->ctl;
    sp.pmax = c->pmax;
    sp.pidx = c->pidx;
    sp.n_wg = c->n_wg_lm;
    sp.out = out_dev;
    sp.stream = stream_dev;
    if (with_lm) {
        GemmParams lm = base;
        lm.W = c->w_lm;
        lm.Ks = c->ks_d;
        lm.n_wg = c->n_wg_lm;
        lm.A = c->An;
        lm.lda = c->d;
        lm.pmax = c->pmax;
        lm.pidx = c->pidx;
        lm.dbg = c->dbg_on ? c->dbg : nullptr;
        timing_events(c, CLLM_KT_LM_HEAD, rg, &e0, &e1);
        HIPCHK(c, launch_gemm(GEMM_LM, c->bf16, rg, lm, s, e0, e1));
        sp.advance_only = 0;
    } else {
        sp.advance_only = 1;
    }
    timing_events(c, CLLM_KT_SCAN, rg, &e0, &e1);
    HIPCHK(c, launch_scan(sp, s, e0, e1));
    return CLLM_OK;
}

cllm_status setup(cllm_ctx *c, int mode, int m, const int32_t *z, bool set_L, int L) {
    SetupParams sp{};
    sp.ctl = c->ctl;
    sp.mode = mode;
    sp.m = m;
    sp.set_L = set_L ? 1 : 0;
    sp.L = L;
    for (int i = 0; i < m; ++i) sp.z[i] = z[i];
    HIPCHK(c, launch_setup(sp, c->stream));
    return CLLM_OK;
}

cllm_status read_ctl(cllm_ctx *c, Ctl *h) {
    HIPCHK(c, hipMemcpyAsync(h, c->ctl, sizeof(Ctl), hipMemcpyDeviceToHost, c->stream));
    HIPCHK(c, hipStreamSynchronize(c->stream));
    if (c->kt_class >= 0) timing_collect(c);
    return CLLM_OK;
}

cllm_status check_ids(cllm_ctx *c, const int32_t *ids, int n) {
    for (int i = 0; i < n; ++i)
        if (ids[i] < 0 || ids[i] >= c->V) return fail(c, CLLM_ERR_ARG, "token id %d at index %d out of range", ids[i], i);
    return CLLM_OK;
}

cllm_status prefill_impl(cllm_ctx *c, const int32_t *prompt, int len, int nch_launch_extra) {
    c->prefilled = false;
    const int nchunks = (len + kMaxRows - 1) / kMaxRows;
    for (int k = 0; k < nchunks; ++k) {
        const int start = k * kMaxRows;
        const int rows = std::min(kMaxRows, len - start);
        cllm_status st = setup(c, MODE_PREFILL, rows, prompt + start, k == 0, 0);
        if (st) return st;
        const int nch = std::min(c->nch, (start + rows + kAttnChunk - 1) / kAttnChunk);
        st = enqueue_iteration(c, rows, nch, k == nchunks - 1, nullptr, nullptr);
        if (st) return st;
    }
    (void)nch_launch_extra;
    return CLLM_OK;
}

}  // namespace

// ------------------------------------------------------------------------------------------
// C ABI
// ------------------------------------------------------------------------------------------
extern "C" {

const char *cllm_status_string(cllm_status s) {
    switch (s) {
    case CLLM_OK: return "ok";
    case CLLM_ERR_ARG: return "invalid argument";
    case CLLM_ERR_STATE: return "invalid state";
    case CLLM_ERR_CAPACITY: return "capacity exceeded";
    case CLLM_ERR_OOM: return "out of memory";
    case CLLM_ERR_IO: return "i/o error";
    case CLLM_ERR_FORMAT: return "bad weight file";
    case CLLM_ERR_DEVICE: return "device error";
    case CLLM_ERR_NUMERIC: return "NaN logit";
    }
    return "unknown status";
}

const char *cllm_last_error(const cllm_ctx *ctx) { return ctx ? ctx->err.c_str() : "null context"; }

int64_t cllm_streamed_weight_bytes(const cllm_ctx *ctx) { return ctx ? ctx->streamed_bytes : 0; }

void cllm_model_free(cllm_ctx *c) {
    if (!c) return;
    if (c->stream) (void)hipStreamSynchronize(c->stream);
    for (void *p : c->allocs) (void)hipFree(p);
    for (hipEvent_t e : c->ev_pool) (void)hipEventDestroy(e);
    delete c;
}

cllm_status cllm_model_create(const cllm_config *cfg, const cllm_runtime_opts *opts, cllm_ctx **out) {
    if (!cfg || !opts || !out) return CLLM_ERR_ARG;
    *out = nullptr;
    const bool bf16 = cfg->dtype == CLLM_DTYPE_BF16;
    const int kstep = bf16 ? 32 : 16;
    if ((cfg->dtype != CLLM_DTYPE_BF16 && cfg->dtype != CLLM_DTYPE_F32) || cfg->n_layers < 1 || cfg->d_model < 1 ||
        cfg->n_heads < 1 || cfg->n_heads * cfg->head_dim != cfg->d_model ||
        !(cfg->head_dim == 32 || cfg->head_dim == 64 || cfg->head_dim == 128 ||
          (bf16 ? cfg->head_dim == 256 : cfg->head_dim == 16)) ||
        cfg->d_model % 64 != 0 || cfg->d_model > 8192 ||
        cfg->ffn_dim < 1 || cfg->vocab < 2 || !(cfg->rms_eps >= 0.0f) || !(cfg->rope_base > 0.0f))
        return CLLM_ERR_ARG;
    if (opts->max_block < 1 || opts->max_block > kMaxBlock || opts->max_ctx < 2 ||
        opts->max_ctx > kMaxChunks * kAttnChunk - 2 * kMaxRows || opts->max_new < 1)
        return CLLM_ERR_ARG;
    int ndev = 0;
    if (hipGetDeviceCount(&ndev) != hipSuccess || opts->device < 0 || opts->device >= ndev) {
        (void)hipGetLastError();
        return CLLM_ERR_DEVICE;
    }
    cllm_ctx *c = new (std::nothrow) cllm_ctx;
    if (!c) return CLLM_ERR_OOM;
    c->cfg = *cfg;
    c->opts = *opts;
    c->bf16 = bf16;
    c->elem = bf16 ? 2 : 4;
    c->NL = cfg->n_layers;
    c->d = cfg->d_model;
    c->H = cfg->n_heads;
    c->hd = cfg->head_dim;
    c->F = cfg->ffn_dim;
    c->V = cfg->vocab;
    c->Fp = round_up(c->F, 32);
    c->ctx_alloc = round_up(opts->max_ctx + kMaxRows, kAttnChunk);
    c->nch = c->ctx_alloc / kAttnChunk;
    c->ks_d = c->d / kstep;
    c->ks_f = c->Fp / kstep;
    c->n_wg_qkv = 3 * c->d / 16 / kNtQkv;
    c->n_wg_o = c->d / 16 / kNtResid;
    c->n_wg_gu = 2 * c->Fp / 16 / kNtGateUp;
    c->n_wg_d = c->d / 16 / kNtResid;
    c->n_wg_lm = round_up(c->V, 16 * kLmTiles) / (16 * kLmTiles);
    c->stream = static_cast<hipStream_t>(opts->stream);

    auto bail = [&](cllm_status s) {
        cllm_model_free(c);
        return s;
    };
    if (hipSetDevice(opts->device) != hipSuccess) return bail(CLLM_ERR_DEVICE);
    cllm_status s;
    const size_t E = c->elem;
    const size_t rows = kMaxRows;
    if ((s = dalloc(c, &c->embed, (size_t)c->V * c->d * E))) return bail(s);
    c->g_attn.assign(c->NL, nullptr);
    c->g_ffn.assign(c->NL, nullptr);
    c->w_qkv.assign(c->NL, nullptr);
    c->w_o.assign(c->NL, nullptr);
    c->w_gu.assign(c->NL, nullptr);
    c->w_d.assign(c->NL, nullptr);
    for (int l = 0; l < c->NL; ++l) {
        if ((s = dalloc_t(c, &c->g_attn[l], c->d))) return bail(s);
        if ((s = dalloc_t(c, &c->g_ffn[l], c->d))) return bail(s);
    }
    if ((s = dalloc_t(c, &c->g_final, c->d))) return bail(s);
    const size_t kv = (size_t)c->NL * c->ctx_alloc * c->d * E;
    if ((s = dalloc(c, &c->kc, kv))) return bail(s);
    if ((s = dalloc(c, &c->vt, kv))) return bail(s);
    const int h2 = c->hd / 2;
    if ((s = dalloc_t(c, &c->rcos, (size_t)c->ctx_alloc * h2))) return bail(s);
    if ((s = dalloc_t(c, &c->rsin, (size_t)c->ctx_alloc * h2))) return bail(s);
    if ((s = dalloc_t(c, &c->X, rows * c->d))) return bail(s);
    if ((s = dalloc_t(c, &c->ssq, (size_t)(c->d / 16) * rows))) return bail(s);
    // activation operands: one fp32 plane, or hi and lo bf16 planes (4 bytes per element either way)
    if ((s = dalloc(c, &c->Q, act_plane(c->d) * 4))) return bail(s);
    if ((s = dalloc(c, &c->O, act_plane(c->d) * 4))) return bail(s);
    if ((s = dalloc(c, &c->An, act_plane(c->d) * 4))) return bail(s);
    if ((s = dalloc(c, &c->Hb, act_plane(c->Fp) * 4))) return bail(s);
    if ((s = dalloc_t(c, &c->pmax, (size_t)c->n_wg_lm * rows))) return bail(s);
    if ((s = dalloc_t(c, &c->pidx, (size_t)c->n_wg_lm * rows))) return bail(s);
    if ((s = dalloc_t(c, &c->opart, (size_t)c->H * c->nch * rows * c->hd))) return bail(s);
    if ((s = dalloc_t(c, &c->mpart, (size_t)c->H * c->nch * rows))) return bail(s);
    if ((s = dalloc_t(c, &c->lpart, (size_t)c->H * c->nch * rows))) return bail(s);
    if ((s = dalloc_t(c, &c->dbg, rows * c->V))) return bail(s);
    if ((s = dalloc_t(c, &c->ctl, 1))) return bail(s);
    if ((s = dalloc_t(c, &c->out_dev, (size_t)opts->max_new))) return bail(s);
    c->stream_cap = opts->max_new + kMaxBlock;
    if ((s = dalloc_t(c, &c->stream_dev, (size_t)c->stream_cap))) return bail(s);

    // RoPE table: angle t * base^(-2j/hd) in double, rounded once to fp32.
    std::vector<float> hc((size_t)c->ctx_alloc * h2), hs((size_t)c->ctx_alloc * h2);
    for (int t = 0; t < c->ctx_alloc; ++t)
        for (int j = 0; j < h2; ++j) {
            const double ang = (double)t * std::pow((double)cfg->rope_base, -2.0 * j / (double)c->hd);
            hc[(size_t)t * h2 + j] = (float)std::cos(ang);
            hs[(size_t)t * h2 + j] = (float)std::sin(ang);
        }
    if (hipMemcpy(c->rcos, hc.data(), hc.size() * 4, hipMemcpyHostToDevice) != hipSuccess ||
        hipMemcpy(c->rsin, hs.data(), hs.size() * 4, hipMemcpyHostToDevice) != hipSuccess)
        return bail(CLLM_ERR_DEVICE);
    // Packed weight buffers (zero until set_weights).
    const int lm_rows = round_up(c->V, 16 * kLmTiles);
    c->streamed_bytes = 0;
    auto packed = [&](uint8_t **dst, int n_rows, int K) -> cllm_status {
        const int Ks = round_up(K, kstep) / kstep;
        const size_t bytes = (size_t)(n_rows / 16) * Ks * kTileBytes;
        c->streamed_bytes += (int64_t)bytes;
        return dalloc(c, reinterpret_cast<void **>(dst), bytes);
    };
    for (int l = 0; l < c->NL; ++l) {
        if ((s = packed(&c->w_qkv[l], 3 * c->d, c->d))) return bail(s);
        if ((s = packed(&c->w_o[l], c->d, c->d))) return bail(s);
        if ((s = packed(&c->w_gu[l], 2 * c->Fp, c->d))) return bail(s);
        if ((s = packed(&c->w_d[l], c->d, c->Fp))) return bail(s);  // Fp is a multiple of both k-steps
    }
    if ((s = packed(&c->w_lm, lm_rows, c->d))) return bail(s);
    if (hipStreamSynchronize(c->stream) != hipSuccess) return bail(CLLM_ERR_DEVICE);
    *out = c;
    return CLLM_OK;
}

cllm_status cllm_model_set_weights(cllm_ctx *c, const void *const *tensors, int32_t n_tensors) {
    if (!c) return CLLM_ERR_ARG;
    if (c->dead) return fail(c, CLLM_ERR_DEVICE, "context unusable after a device error: %s", c->err.c_str());
    if (!tensors || n_tensors != 3 + 9 * c->NL) return fail(c, CLLM_ERR_ARG, "expected %d tensors", 3 + 9 * c->NL);
    for (int i = 0; i < n_tensors; ++i)
        if (!tensors[i]) return fail(c, CLLM_ERR_ARG, "tensor %d is NULL", i);
    const int d = c->d, F = c->F, V = c->V;
    const size_t E = c->elem;
    size_t stage_elems = std::max({(size_t)3 * d * d, (size_t)2 * F * d, (size_t)V * d});
    void *staging = nullptr;
    int32_t *perm_dev = nullptr;
    if (hipMalloc(&staging, stage_elems * E) != hipSuccess) {
        (void)hipGetLastError();
        return fail(c, CLLM_ERR_OOM, "staging allocation failed");
    }
    const size_t perm_max = std::max({(size_t)3 * d, (size_t)2 * c->Fp, (size_t)round_up(V, 16 * kLmTiles)});
    if (hipMalloc(reinterpret_cast<void **>(&perm_dev), perm_max * 4) != hipSuccess) {
        (void)hipGetLastError();
        (void)hipFree(staging);
        return fail(c, CLLM_ERR_OOM, "staging allocation failed");
    }
    std::vector<uint8_t> cat;
    cllm_status s = CLLM_OK;
    auto gain = [&](float *dst, const void *src) -> cllm_status {
        HIPCHK(c, hipMemcpyAsync(dst, src, (size_t)d * 4, hipMemcpyHostToDevice, c->stream));
        return CLLM_OK;
    };
    const std::vector<int32_t> pq = qkv_perm(c), pgu = gate_up_perm(c), pd = plain_perm(d, d),
                               plm = plain_perm(round_up(V, 16 * kLmTiles), V);
    c->streamed_bytes = 0;
    do {
        if (hipMemcpyAsync(c->embed, tensors[0], (size_t)V * d * E, hipMemcpyHostToDevice, c->stream) != hipSuccess) {
            s = fail(c, CLLM_ERR_DEVICE, "embedding upload failed");
            break;
        }
        for (int l = 0; l < c->NL && !s; ++l) {
            const void *const *t = tensors + 1 + 9 * l;
            if ((s = gain(c->g_attn[l], t[0]))) break;
            cat.resize((size_t)3 * d * d * E);
            for (int k = 0; k < 3; ++k) memcpy(cat.data() + (size_t)k * d * d * E, t[1 + k], (size_t)d * d * E);
            if ((s = upload_packed(c, cat.data(), 3 * d, d, c->ks_d, pq, &c->w_qkv[l], staging, perm_dev))) break;
            if ((s = upload_packed(c, t[4], d, d, c->ks_d, pd, &c->w_o[l], staging, perm_dev))) break;
            if ((s = gain(c->g_ffn[l], t[5]))) break;
            cat.resize((size_t)2 * F * d * E);
            memcpy(cat.data(), t[6], (size_t)F * d * E);
            memcpy(cat.data() + (size_t)F * d * E, t[7], (size_t)F * d * E);
            if ((s = upload_packed(c, cat.data(), 2 * F, d, c->ks_d, pgu, &c->w_gu[l], staging, perm_dev))) break;
            if ((s = upload_packed(c, t[8], d, F, c->ks_f, pd, &c->w_d[l], staging, perm_dev))) break;
        }
        if (s) break;
        if ((s = gain(c->g_final, tensors[1 + 9 * c->NL]))) break;
        if ((s = upload_packed(c, tensors[2 + 9 * c->NL], V, d, c->ks_d, plm, &c->w_lm, staging, perm_dev))) break;
    } while (0);
    hipError_t e = hipStreamSynchronize(c->stream);
    (void)hipFree(staging);
    (void)hipFree(perm_dev);
    if (s) return s;
    if (e != hipSuccess) return fail(c, CLLM_ERR_DEVICE, "weight upload failed: %s", hipGetErrorString(e));
    c->prefilled = false;
    return CLLM_OK;
}

cllm_status cllm_model_load(const char *path, const cllm_runtime_opts *opts, cllm_ctx **out) {
    if (!path || !opts || !out) return CLLM_ERR_ARG;
    *out = nullptr;
    FILE *f = fopen(path, "rb");
    if (!f) return CLLM_ERR_IO;
    unsigned char hdr[64];
    if (fread(hdr, 1, 64, f) != 64) {
        fclose(f);
        return CLLM_ERR_FORMAT;
    }
    int32_t version;
    cllm_config cfg;
    memcpy(&version, hdr + 8, 4);
    memcpy(&cfg.n_layers, hdr + 12, 4);
    memcpy(&cfg.d_model, hdr + 16, 4);
    memcpy(&cfg.n_heads, hdr + 20, 4);
    memcpy(&cfg.head_dim, hdr + 24, 4);
    memcpy(&cfg.ffn_dim, hdr + 28, 4);
    memcpy(&cfg.vocab, hdr + 32, 4);
    memcpy(&cfg.rms_eps, hdr + 36, 4);
    memcpy(&cfg.rope_base, hdr + 40, 4);
    memcpy(&cfg.dtype, hdr + 44, 4);
    if (memcmp(hdr, "CLLMWTS1", 8) != 0 || version != 1 || cfg.n_layers < 1 || cfg.n_layers > 4096 ||
        cfg.d_model < 1 || cfg.d_model > (1 << 16) || cfg.ffn_dim < 1 || cfg.ffn_dim > (1 << 18) || cfg.vocab < 2 ||
        cfg.vocab > (1 << 22)) {
        fclose(f);
        return CLLM_ERR_FORMAT;
    }
    cllm_ctx *c = nullptr;
    cllm_status s = cllm_model_create(&cfg, opts, &c);
    if (s) {
        fclose(f);
        return s == CLLM_ERR_ARG ? CLLM_ERR_FORMAT : s;
    }
    const size_t E = cfg.dtype == CLLM_DTYPE_BF16 ? 2 : 4;
    const size_t d = cfg.d_model, F = cfg.ffn_dim, V = cfg.vocab;
    std::vector<size_t> sizes;
    sizes.push_back(V * d * E);
    for (int l = 0; l < cfg.n_layers; ++l) {
        sizes.push_back(d * 4);
        for (int k = 0; k < 4; ++k) sizes.push_back(d * d * E);
        sizes.push_back(d * 4);
        sizes.push_back(F * d * E);
        sizes.push_back(F * d * E);
        sizes.push_back(d * F * E);
    }
    sizes.push_back(d * 4);
    sizes.push_back(V * d * E);
    std::vector<std::vector<uint8_t>> bufs(sizes.size());
    std::vector<const void *> ptrs(sizes.size());
    for (size_t i = 0; i < sizes.size(); ++i) {
        bufs[i].resize(sizes[i]);
        if (fread(bufs[i].data(), 1, sizes[i], f) != sizes[i]) {
            fclose(f);
            cllm_model_free(c);
            return CLLM_ERR_FORMAT;
        }
        ptrs[i] = bufs[i].data();
    }
    unsigned char extra;
    const bool trailing = fread(&extra, 1, 1, f) == 1;
    fclose(f);
    if (trailing) {
        cllm_model_free(c);
        return CLLM_ERR_FORMAT;
    }
    s = cllm_model_set_weights(c, ptrs.data(), (int32_t)ptrs.size());
    if (s) {
        cllm_model_free(c);
        return s;
    }
    *out = c;
    return CLLM_OK;
}

cllm_status cllm_prefill(cllm_ctx *c, int32_t seq, const int32_t *prompt, int32_t len, int32_t *first_token) {
    if (!c) return CLLM_ERR_ARG;
    if (c->dead) return fail(c, CLLM_ERR_DEVICE, "context unusable after a device error: %s", c->err.c_str());
    if (seq != 0) return fail(c, CLLM_ERR_ARG, "seq must be 0");
    if (!prompt || !first_token || len < 1) return fail(c, CLLM_ERR_ARG, "bad prompt");
    if (len + 1 > c->opts.max_ctx) return fail(c, CLLM_ERR_CAPACITY, "prompt of %d exceeds max_ctx", len);
    cllm_status s;
    if ((s = check_ids(c, prompt, len))) return s;
    if ((s = prefill_impl(c, prompt, len, 0))) return s;
    Ctl h;
    if ((s = read_ctl(c, &h))) return s;
    if (h.err) return fail(c, CLLM_ERR_NUMERIC, "NaN logit in the prefill");
    if (c->dbg_on && c->dbg_host) {
        const int rows = len - (len - 1) / kMaxRows * kMaxRows;
        HIPCHK(c, hipMemcpy(c->dbg_host, c->dbg, (size_t)rows * c->V * 4, hipMemcpyDeviceToHost));
    }
    c->prefilled = true;
    c->L = h.L;
    c->pending = h.pending;
    *first_token = h.pending;
    return CLLM_OK;
}

cllm_status cllm_jacobi_step(cllm_ctx *c, int32_t seq, const int32_t *block_in, int32_t m, int32_t *block_out,
                             int32_t *accepted_len) {
    if (!c) return CLLM_ERR_ARG;
    if (c->dead) return fail(c, CLLM_ERR_DEVICE, "context unusable after a device error: %s", c->err.c_str());
    if (seq != 0) return fail(c, CLLM_ERR_ARG, "seq must be 0");
    if (!block_in || !block_out || !accepted_len) return fail(c, CLLM_ERR_ARG, "NULL pointer");
    if (m < 1 || m > c->opts.max_block) return fail(c, CLLM_ERR_ARG, "m=%d outside [1, max_block]", m);
    if (!c->prefilled) return fail(c, CLLM_ERR_STATE, "jacobi_step before prefill");
    cllm_status s;
    if ((s = check_ids(c, block_in, m))) return s;
    if (block_in[0] != c->pending)
        return fail(c, CLLM_ERR_STATE, "block_in[0]=%d is not the pending token %d", block_in[0], c->pending);
    if (c->L + m > c->opts.max_ctx) return fail(c, CLLM_ERR_CAPACITY, "L + m exceeds max_ctx");
    if ((s = setup(c, MODE_STEP, m, block_in, false, 0))) return s;
    const int nch = (c->L + m + kAttnChunk - 1) / kAttnChunk;
    if ((s = enqueue_iteration(c, m, nch, true, nullptr, nullptr))) return s;
    Ctl h;
    if ((s = read_ctl(c, &h))) return s;
    if (h.err) return fail(c, CLLM_ERR_NUMERIC, "NaN logit");
    if (c->dbg_on && c->dbg_host) HIPCHK(c, hipMemcpy(c->dbg_host, c->dbg, (size_t)m * c->V * 4, hipMemcpyDeviceToHost));
    for (int i = 0; i < m; ++i) block_out[i] = h.pred[i];
    *accepted_len = h.a_last;
    c->L = h.L;
    c->pending = h.pending;
    return CLLM_OK;
}

static cllm_status decode_impl(cllm_ctx *c, const int32_t *prompt, int32_t len, int32_t n, int32_t max_new,
                               const cllm_guess_spec *g, int32_t *out_tokens, cllm_decode_stats *stats) {
    if (!prompt || !out_tokens || len < 1) return fail(c, CLLM_ERR_ARG, "bad prompt or output");
    if (n < 1 || n > c->opts.max_block) return fail(c, CLLM_ERR_ARG, "n=%d outside [1, max_block]", n);
    if (max_new < 1) return fail(c, CLLM_ERR_ARG, "max_new must be >= 1");
    if (max_new > c->opts.max_new) return fail(c, CLLM_ERR_CAPACITY, "max_new exceeds the context's max_new");
    if (len + max_new + n > c->opts.max_ctx) return fail(c, CLLM_ERR_CAPACITY, "len + max_new + n exceeds max_ctx");
    cllm_guess_spec gs{};
    if (g) gs = *g;
    if (gs.policy < 0 || gs.policy > 2 || gs.block_policy < 0 || gs.block_policy > 1)
        return fail(c, CLLM_ERR_ARG, "bad guess policy");
    if (gs.policy != CLLM_GUESS_UNIFORM) {
        if (!gs.stream || gs.stream_len < max_new) return fail(c, CLLM_ERR_ARG, "guess stream shorter than max_new");
        if (gs.thr53 > (1ull << 53)) return fail(c, CLLM_ERR_ARG, "thr53 above 2^53");
    }
    cllm_status s;
    if ((s = check_ids(c, prompt, len))) return s;
    if (gs.policy != CLLM_GUESS_UNIFORM && (s = check_ids(c, gs.stream, max_new))) return s;

    hipEvent_t ev[3];
    for (auto &e : ev) HIPCHK(c, hipEventCreate(&e));
    struct EvGuard {
        hipEvent_t *e;
        ~EvGuard() {
            for (int i = 0; i < 3; ++i) (void)hipEventDestroy(e[i]);
        }
    } guard{ev};

    if (gs.policy != CLLM_GUESS_UNIFORM)
        HIPCHK(c, hipMemcpyAsync(c->stream_dev, gs.stream, (size_t)max_new * 4, hipMemcpyHostToDevice, c->stream));
    HIPCHK(c, hipEventRecord(ev[0], c->stream));
    if ((s = prefill_impl(c, prompt, len, 0))) return s;
    HIPCHK(c, hipEventRecord(ev[1], c->stream));
    // Decode parameters into the control block (the prefill left L and pending there).
    Ctl h;
    if ((s = read_ctl(c, &h))) return s;
    if (h.err) return fail(c, CLLM_ERR_NUMERIC, "NaN logit in the prefill");
    h.n = n;
    h.max_new = max_new;
    h.policy = gs.policy;
    h.block_policy = gs.block_policy;
    h.seq = 0;
    h.stream_len = gs.policy != CLLM_GUESS_UNIFORM ? max_new : 0;
    h.vocab = c->V;
    h.seed = gs.seed;
    h.thr53 = gs.thr53;
    HIPCHK(c, hipMemcpyAsync(c->ctl, &h, sizeof(Ctl), hipMemcpyHostToDevice, c->stream));
    ScanParams sp{};
    sp.ctl = c->ctl;
    sp.stream = gs.policy != CLLM_GUESS_UNIFORM ? c->stream_dev : nullptr;
    HIPCHK(c, launch_decode_init(sp, c->stream));
    const int nch = std::min(c->nch, (len + max_new + n + kAttnChunk - 1) / kAttnChunk);
    // Device-resident loop: every launch reads its block from the control block. The host only
    // queues iterations; it queues as many as are certainly needed (each iteration fixes at most
    // n tokens) and then reads the emitted count once.
    int emitted = 0;
    int64_t guard_iters = 0;
    while (true) {
        const int need = (max_new - emitted + n - 1) / n;
        for (int i = 0; i < need; ++i)
            if ((s = enqueue_iteration(c, n, nch, true, c->out_dev,
                                       gs.policy != CLLM_GUESS_UNIFORM ? c->stream_dev : nullptr)))
                return s;
        guard_iters += need;
        HIPCHK(c, hipEventRecord(ev[2], c->stream));
        if ((s = read_ctl(c, &h))) return s;
        if (h.err) return fail(c, CLLM_ERR_NUMERIC, "NaN logit");
        emitted = h.e;
        if (h.done) break;
        if (guard_iters > (int64_t)max_new + 1) return fail(c, CLLM_ERR_STATE, "decode did not finish");
    }
    HIPCHK(c, hipMemcpy(out_tokens, c->out_dev, (size_t)max_new * 4, hipMemcpyDeviceToHost));
    if (stats) {
        memset(stats, 0, sizeof(*stats));
        stats->steps = h.steps;
        stats->blocks = h.blocks;
        stats->tokens = h.e;
        for (int i = 0; i <= kMaxBlock; ++i) stats->accept_hist[i] = h.hist[i];
        float ms = 0.f;
        if (hipEventElapsedTime(&ms, ev[0], ev[1]) == hipSuccess) stats->prefill_ms = ms;
        if (hipEventElapsedTime(&ms, ev[1], ev[2]) == hipSuccess) stats->decode_ms = ms;
    }
    c->prefilled = true;
    c->L = h.L;
    c->pending = h.pending;
    return CLLM_OK;
}

cllm_status cllm_jacobi_decode(cllm_ctx *c, int32_t seq, const int32_t *prompt, int32_t len, int32_t n,
                               int32_t max_new, const cllm_guess_spec *guess, int32_t *out_tokens,
                               cllm_decode_stats *stats) {
    if (!c) return CLLM_ERR_ARG;
    if (c->dead) return fail(c, CLLM_ERR_DEVICE, "context unusable after a device error: %s", c->err.c_str());
    if (seq != 0) return fail(c, CLLM_ERR_ARG, "seq must be 0");
    return decode_impl(c, prompt, len, n, max_new, guess, out_tokens, stats);
}

cllm_status cllm_ar_decode(cllm_ctx *c, int32_t seq, const int32_t *prompt, int32_t len, int32_t max_new,
                           int32_t *out_tokens, cllm_decode_stats *stats) {
    if (!c) return CLLM_ERR_ARG;
    if (c->dead) return fail(c, CLLM_ERR_DEVICE, "context unusable after a device error: %s", c->err.c_str());
    if (seq != 0) return fail(c, CLLM_ERR_ARG, "seq must be 0");
    cllm_guess_spec g{};
    return decode_impl(c, prompt, len, 1, max_new, &g, out_tokens, stats);
}

cllm_status cllm_debug_logits(cllm_ctx *c, int32_t enable, float *host_buf, size_t host_floats) {
    if (!c) return CLLM_ERR_ARG;
    if (enable) {
        if (!host_buf || host_floats < (size_t)std::max(c->opts.max_block, kMaxRows) * c->V)
            return fail(c, CLLM_ERR_ARG, "debug buffer needs %zu floats", (size_t)std::max(c->opts.max_block, kMaxRows) * c->V);
        c->dbg_on = true;
        c->dbg_host = host_buf;
        c->dbg_cap = host_floats;
    } else {
        c->dbg_on = false;
        c->dbg_host = nullptr;
        c->dbg_cap = 0;
    }
    return CLLM_OK;
}

cllm_status cllm_seq_state(const cllm_ctx *c, int32_t seq, int32_t *committed_len, int32_t *pending) {
    if (!c || seq != 0 || !committed_len || !pending) return CLLM_ERR_ARG;
    if (!c->prefilled) return CLLM_ERR_STATE;
    *committed_len = c->L;
    *pending = c->pending;
    return CLLM_OK;
}

cllm_status cllm_timing_enable(cllm_ctx *c, int32_t kernel_class, int32_t max_rows) {
    if (!c) return CLLM_ERR_ARG;
    if (kernel_class > CLLM_KT_EMBED || max_rows < 0 || max_rows > kMaxRows)
        return fail(c, CLLM_ERR_ARG, "unknown kernel class or bad max_rows");
    c->kt_class = kernel_class < 0 ? -1 : kernel_class;
    c->kt_rg = max_rows == 0 ? 0 : rows_to_rg(max_rows);
    c->ev_used = 0;
    c->kt_launches = 0;
    c->kt_ms = 0.0;
    return CLLM_OK;
}

cllm_status cllm_timing_read(cllm_ctx *c, int64_t *launches, double *total_ms) {
    if (!c || !launches || !total_ms) return CLLM_ERR_ARG;
    if (c->ev_used) {
        HIPCHK(c, hipStreamSynchronize(c->stream));
        timing_collect(c);
    }
    *launches = c->kt_launches;
    *total_ms = c->kt_ms;
    c->kt_launches = 0;
    c->kt_ms = 0.0;
    return CLLM_OK;
}

}  // extern "C"
