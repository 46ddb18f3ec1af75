// Runtime of libcllm.so: device memory, weight repacking, the iteration launch sequence, the
// device-resident decode loop and the C ABI of include/cllm.h.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
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
    int n_wg_lm = 0;  // LM-head workgroups (argmax partials per row)
    int max_batch = 1;
    int cap = 0;        // row capacity of one iteration (multiple of 64): activation buffer rows
    int pchunk = 0;     // prompt rows per prefill pass (multiple of 64, <= cap)
    int dbg_rows = 0;   // rows of a step's debug logits: max(64, max_batch * max_block) rounded up
    size_t kv_seq = 0;  // KV cache elements per sequence slot
    int64_t streamed_bytes = 0;

    // weights
    void *embed = nullptr;
    std::vector<float *> g_attn, g_ffn;
    float *g_final = nullptr;
    std::vector<uint8_t *> w_qkv, w_o, w_gu, w_d;
    uint8_t *w_lm = nullptr;
    // KV cache per slot: K [slot][layer][ctx_alloc][d], V transposed [slot][layer][d][ctx_alloc]
    void *kc = nullptr, *vt = nullptr;
    float *rcos = nullptr, *rsin = nullptr;
    // workspace
    float *part = nullptr;  // K-split partial products of the down projection: kDownSplits x rows x d
    float *spart = nullptr;  // class-pair split partials of multi-row products (bf16): 4 x rows x max columns
    float *sinv = nullptr;   // their RMSNorm row factors: rows
    float *X = nullptr, *ssq = nullptr, *pmax = nullptr, *opart = nullptr, *mpart = nullptr, *lpart = nullptr,
          *dbg = nullptr;
    int *pidx = nullptr;
    void *Q = nullptr, *O = nullptr, *Hb = nullptr;
    void *An = nullptr;  // RMSNorm operand x (.) g of the next normed product
    Ctl *ctl = nullptr;  // one control block per slot
    RowTab *tab = nullptr;
    RowInfo *rows = nullptr;
    int32_t *zin = nullptr;  // staging of host tokens (blocks, prefill chunks)
    int zin_cap = 0;
    int32_t *out_dev = nullptr, *stream_dev = nullptr;  // per slot: max_new outputs, stream_cap guesses
    int32_t *mlog_dev = nullptr;  // per slot: block size of each decode iteration (max_new entries)
    std::vector<hipEvent_t> it_ev;  // one per queued decode iteration
    // decode loop: the control blocks as they stand before a round's last iteration (pinned
    // host memory, read while that iteration runs) and the event after their copy
    Ctl *ctl_snap = nullptr;
    hipEvent_t snap_ev = nullptr;
    int stream_cap = 0;
    std::vector<void *> allocs;
    // caller-owned workspace (cllm_runtime_opts.workspace): the iteration buffers are carved from
    // it instead of being allocated; it is never freed by the library
    uint8_t *ws_base = nullptr;
    size_t ws_size = 0, ws_off = 0;

    // host state per slot
    struct Slot {
        bool prefilled = false;
        // a NaN logit was reported: the cache may hold NaN rows past the committed length, which a
        // later request's attention would multiply by zero probabilities (giving NaN), so the
        // slot's next prefill clears its cache first
        bool dirty = false;
        int L = 0, pending = 0;
        int64_t trace_n = 0;  // trajectory records of the slot's last recorded decode
    };
    int32_t *trace_dev = nullptr;  // trajectory records: max_batch x max_new x kTraceStride int32
    bool trace_on = false;
    // loss head workspace (allocated on first use, grown on demand)
    struct LossWs {
        size_t h = 0, a = 0, z = 0, dd = 0, part = 0, dh = 0, dw = 0, rows = 0, st = 0, da = 0, dt = 0, ht = 0;
        float *H = nullptr, *Z = nullptr, *D = nullptr, *part_p = nullptr, *dH = nullptr, *dW = nullptr,
              *out = nullptr, *stats = nullptr;
        uint8_t *A = nullptr;     // GEMM operand planes of the input rows (bytes)
        uint8_t *Dact = nullptr;  // GEMM operand planes of D (bytes)
        uint16_t *DT = nullptr, *HT = nullptr;  // dW operands (bf16 planes)
        uint8_t *WT = nullptr;    // the packed LM head transposed (built on first use)
        bool wt_ok = false;       // WT holds the current LM head
        int32_t *tg = nullptr;
        RowTab *tabs = nullptr;   // row tables of the loss GEMMs: tabs[R - 1] holds R rows (R <= 128)
        double *loss = nullptr;   // staging of the host entry point's total
        float *hid = nullptr;     // LM-head input rows of cllm_hidden_rows
        size_t hd_n = 0;
    } loss;
    std::vector<Slot> slot;
    bool dead = false;
    std::string err;
    bool dbg_on = false;
    float *dbg_host = nullptr;
    size_t dbg_cap = 0;
    // kernel timing
    int kt_class = -1;
    int kt_rg = 0;  // time only launches for this many 16-row groups (0 = all)
    int kt_every = 1;           // time one of every kt_every eligible launches
    int64_t kt_eligible = 0;    // eligible launches since the last enable
    bool in_prefill = false;  // prefill launches are not timed
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

static_assert(CLLM_TRACE_STRIDE == kTraceStride && kMaxBlock == 64, "trajectory record layout of the header");

inline int round_up(int x, int a) { return (x + a - 1) / a * a; }
inline int rows_to_rg(int rows) { return rows <= 16 ? 1 : (rows <= 32 ? 2 : 4); }
inline int ceil_div(int a, int b) { return (a + b - 1) / b; }

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

// The iteration workspace of a context: activation operands, split and attention partials,
// argmax partials, control blocks, the row table, token staging and decode outputs (every buffer
// made at creation except the weights, the RoPE tables and the KV cache). Each buffer starts at a
// 256-byte boundary.
struct WsBuf {
    void **p;
    size_t bytes;
};
constexpr size_t kWsAlign = 256;

std::vector<WsBuf> workspace_bufs(cllm_ctx *c) {
    const size_t rows = c->cap, d = c->d;
    const size_t mb = c->max_batch, max_new = c->opts.max_new;
    c->zin_cap = std::max(c->cap, c->max_batch * c->opts.max_block);
    c->stream_cap = c->opts.max_new + kMaxBlock;
    auto P = [](auto **q) { return reinterpret_cast<void **>(q); };
    // activation operands: one fp32 plane, or hi and lo bf16 planes (4 bytes per element either way)
    return {
        {P(&c->X), rows * d * 4},
        {P(&c->part), (size_t)kDownSplits * rows * d * 4},
        {P(&c->spart), c->bf16 ? 4 * rows * std::max({3 * d, 2 * (size_t)c->Fp, (size_t)c->n_wg_lm * 16 * kLmTiles}) * 4
                               : 16},
        {P(&c->sinv), rows * 4},
        {P(&c->ssq), (d / 16) * rows * 4},
        {P(&c->Q), act_plane(c->cap, c->d) * 4},
        {P(&c->O), act_plane(c->cap, c->d) * 4},
        {P(&c->An), act_plane(c->cap, c->d) * 4},
        {P(&c->Hb), act_plane(c->cap, c->Fp) * 4},
        {P(&c->pmax), (size_t)c->n_wg_lm * rows * 4},
        {P(&c->pidx), (size_t)c->n_wg_lm * rows * 4},
        {P(&c->opart), (size_t)c->H * c->nch * rows * c->hd * 4},
        {P(&c->mpart), (size_t)c->H * c->nch * rows * 4},
        {P(&c->lpart), (size_t)c->H * c->nch * rows * 4},
        {P(&c->ctl), mb * sizeof(Ctl)},
        {P(&c->tab), sizeof(RowTab)},
        {P(&c->rows), rows * sizeof(RowInfo)},
        {P(&c->zin), (size_t)c->zin_cap * 4},
        {P(&c->out_dev), max_new * mb * 4},
        {P(&c->mlog_dev), max_new * mb * 4},
        {P(&c->stream_dev), (size_t)c->stream_cap * mb * 4},
    };
}

size_t workspace_total(const std::vector<WsBuf> &bufs) {
    size_t t = 0;
    for (const WsBuf &b : bufs) t += (std::max<size_t>(b.bytes, 16) + kWsAlign - 1) / kWsAlign * kWsAlign;
    return t;
}

// Place the workspace buffers: carved in order from the caller's buffer when one was given
// (zeroed on the stream), else one hipMalloc each.
cllm_status place_workspace(cllm_ctx *c) {
    const std::vector<WsBuf> bufs = workspace_bufs(c);
    if (!c->ws_base) {
        for (const WsBuf &b : bufs) {
            cllm_status s = dalloc(c, b.p, b.bytes);
            if (s) return s;
        }
        return CLLM_OK;
    }
    const size_t need = workspace_total(bufs);
    if (need > c->ws_size)
        return fail(c, CLLM_ERR_CAPACITY, "workspace of %zu bytes is smaller than the %zu bytes this context needs",
                    c->ws_size, need);
    c->ws_off = 0;
    for (const WsBuf &b : bufs) {
        *b.p = c->ws_base + c->ws_off;
        c->ws_off += (std::max<size_t>(b.bytes, 16) + kWsAlign - 1) / kWsAlign * kWsAlign;
    }
    hipError_t e = hipMemsetAsync(c->ws_base, 0, need, c->stream);
    if (e != hipSuccess) return fail(c, CLLM_ERR_DEVICE, "hipMemsetAsync failed: %s", hipGetErrorString(e));
    return CLLM_OK;
}

// Timing events for the selected kernel class and row-group count (null when not timed).
void timing_events(cllm_ctx *c, int cls, int rg, hipEvent_t *e0, hipEvent_t *e1) {
    *e0 = *e1 = nullptr;
    if (c->kt_class != cls || c->in_prefill || (c->kt_rg > 0 && c->kt_rg != rg && cls < CLLM_KT_LOSS_LOGITS)) return;
    if (c->kt_eligible++ % c->kt_every != 0) return;
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
    for (int R = 0; R < 3 * d; ++R) {  // tile b of a head: dims [8b, 8b+8) and [hd/2+8b, hd/2+8b+8)
        const int sec = R / d, within = R % d, head = within / hd, q = within % hd;
        const int b = q >> 4, o = q & 15;
        const int dim = o < 8 ? 8 * b + o : h2 + 8 * b + (o - 8);
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

// Packs the row-major [N][K] matrix in `staging` into the streaming layout at *dst (perm: the
// logical row of each packed row, -1 = zero). Ks is the k-step count of the packed layout (K
// rounded up; the padding is zero).
cllm_status pack_staged(cllm_ctx *c, int K, int Ks, const std::vector<int32_t> &perm, uint8_t **dst, void *staging,
                        int32_t *perm_dev) {
    const int n_tiles = (int)perm.size() / 16;
    const size_t bytes = (size_t)n_tiles * Ks * kTileBytes;
    if (!*dst) {
        cllm_status s = dalloc(c, reinterpret_cast<void **>(dst), bytes);
        if (s) return s;
    }
    HIPCHK(c, hipMemcpyAsync(perm_dev, perm.data(), perm.size() * sizeof(int32_t), hipMemcpyHostToDevice, c->stream));
    HIPCHK(c, launch_repack(c->bf16, staging, perm_dev, K, Ks, n_tiles, *dst, c->stream));
    HIPCHK(c, hipStreamSynchronize(c->stream));  // staging and perm are reused
    c->streamed_bytes += (int64_t)bytes;
    return CLLM_OK;
}

// Launch shape of one iteration: at most R rows in total, nseq batch entries, at most maxm rows
// per entry, attention over nch chunks. The row table on the device holds the actual rows.
struct IterShape {
    int R, nseq, maxm, nch;
    bool with_lm;
    int lm_rt0;         // >= 0: the LM head runs only on this 64-row tile (a prefill chunk's last row)
    bool tail = true;   // false: the decoder layers only (no LM head, scan or commit)
    bool prompt = false;  // prompt rows (a prefill chunk): bf16 products take the prompt GEMM
    uint64_t lm_mask = 0;   // != 0: the LM head runs only on these 64-row tiles (packed prefill)
    uint64_t adv_mask = 0;  // prefill entries whose chunk does not end their prompt
};

cllm_status enqueue_iteration(cllm_ctx *c, const IterShape &sh, int32_t *out_dev, const int32_t *stream_dev) {
    const bool tiled = sh.R > kMaxRows;
    const int rg = tiled ? 4 : rows_to_rg(sh.R);
    const int row_tiles = tiled ? ceil_div(sh.R, kMaxRows) : 1;
    // prompt rows of a bf16 model: the LDS-tiled prompt GEMM (every prompt row, any chunk size)
    const bool prompt_gemm = sh.prompt && c->bf16;
    hipStream_t s = c->stream;
    hipEvent_t e0, e1;
    const RowsRef rr{c->tab, c->rows, c->cap};

    EmbedParams ep{c->embed, c->X, c->ssq, c->An, c->g_attn[0], c->d, rr};
    timing_events(c, CLLM_KT_EMBED, rg, &e0, &e1);
    HIPCHK(c, launch_embed(c->bf16, sh.R, ep, s, e0, e1));

    GemmParams base{};
    base.rr = rr;
    base.ssq = c->ssq;
    base.T = c->d / 16;
    base.K = c->d;
    base.eps = c->cfg.rms_eps;
    base.d = c->d;
    base.hd = c->hd;
    base.ctx_alloc = c->ctx_alloc;
    base.kv_seq = c->kv_seq;
    base.rcos = c->rcos;
    base.rsin = c->rsin;
    base.Xout = c->X;
    base.ssq_out = c->ssq;
    base.ldx = c->d;
    base.An = c->An;
    base.part = c->part;
    base.spart = c->bf16 ? c->spart : nullptr;
    base.sinv = c->sinv;
    base.Fp = c->Fp;
    base.V = c->V;

    const int arg = std::min(4, ceil_div(std::max(sh.maxm, 1), 16));
    AttnParams ap{};
    ap.Q = c->Q;
    ap.O = c->O;
    ap.kv_seq = c->kv_seq;
    ap.Opart = c->opart;
    ap.Mpart = c->mpart;
    ap.Lpart = c->lpart;
    ap.d = c->d;
    ap.hd = c->hd;
    ap.n_heads = c->H;
    ap.nch = c->nch;
    ap.ctx_alloc = c->ctx_alloc;
    ap.nrb = ceil_div(std::max(sh.maxm, 1), 16 * (arg == 3 ? 4 : arg));
    ap.scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)c->hd));
    ap.rr = rr;
    const int attn_rg = arg == 3 ? 4 : arg;

    const size_t kv_layer = (size_t)c->ctx_alloc * c->d * c->elem;
    for (int l = 0; l < c->NL; ++l) {
        void *kc = static_cast<uint8_t *>(c->kc) + l * kv_layer;
        void *vt = static_cast<uint8_t *>(c->vt) + l * kv_layer;

        GemmParams q = base;  // operand: attention RMSNorm of X, written by the previous producer
        q.W = c->w_qkv[l];
        q.Ks = c->ks_d;
        q.cols = 3 * c->d;
        q.A = c->An;
        q.lda = c->d;
        q.Q = c->Q;
        q.Kc = kc;
        q.Vt = vt;
        timing_events(c, CLLM_KT_GEMM_QKV, rg, &e0, &e1);
        HIPCHK(c, prompt_gemm ? launch_gemm_prompt(GEMM_QKV, sh.R, q, s, e0, e1)
                              : launch_gemm(GEMM_QKV, c->bf16, rg, row_tiles, q, s, e0, e1));

        ap.Kc = kc;
        ap.Vt = vt;
        timing_events(c, CLLM_KT_ATTN, rg, &e0, &e1);
        // one kernel for one sequence's block (<= 64 rows) over a short context (its slices
        // re-read the head's K from L2); the chunk-parallel pair otherwise, including prompt
        // passes of more than 64 rows, whose row groups would re-read every chunk. Both give
        // bit-identical values.
        if (sh.nseq == 1 && sh.nch <= kFusedChunks && c->hd <= 128 && sh.maxm <= kMaxRows) {
            HIPCHK(c, launch_attn_fused(c->bf16, ceil_div(std::max(sh.maxm, 1), 16), sh.nseq, ap, s, e0, e1));
        } else {
            HIPCHK(c, launch_attn(c->bf16, attn_rg, sh.nch, sh.nseq, ap, s, e0, e1));
            timing_events(c, CLLM_KT_ATTN_COMBINE, rg, &e0, &e1);
            HIPCHK(c, launch_attn_combine(c->bf16, sh.R, ap, s, e0, e1));
        }

        GemmParams o = base;  // X += O W_o^T; writes the FFN RMSNorm operand
        o.W = c->w_o[l];
        o.Ks = c->ks_d;
        o.cols = c->d;
        o.A = c->O;
        o.lda = c->d;
        o.gain = c->g_ffn[l];
        timing_events(c, CLLM_KT_GEMM_O, rg, &e0, &e1);
        HIPCHK(c, prompt_gemm ? launch_gemm_prompt(GEMM_O, sh.R, o, s, e0, e1)
                              : launch_gemm(GEMM_O, c->bf16, rg, row_tiles, o, s, e0, e1));

        GemmParams gu = base;
        gu.W = c->w_gu[l];
        gu.Ks = c->ks_d;
        gu.cols = 2 * c->Fp;
        gu.A = c->An;
        gu.lda = c->d;
        gu.H = c->Hb;
        timing_events(c, CLLM_KT_GEMM_GATE_UP, rg, &e0, &e1);
        HIPCHK(c, prompt_gemm ? launch_gemm_prompt(GEMM_GATE_UP, sh.R, gu, s, e0, e1)
                              : launch_gemm(GEMM_GATE_UP, c->bf16, rg, row_tiles, gu, s, e0, e1));

        GemmParams dn = base;  // X += H W_d^T; writes the next layer's (or the final) RMSNorm operand
        dn.W = c->w_d[l];
        dn.Ks = c->ks_f;
        dn.cols = c->d;
        dn.A = c->Hb;
        dn.lda = c->Fp;
        dn.gain = l + 1 < c->NL ? c->g_attn[l + 1] : c->g_final;
        timing_events(c, CLLM_KT_GEMM_DOWN, rg, &e0, &e1);
        HIPCHK(c, prompt_gemm ? launch_gemm_prompt(GEMM_DOWN, sh.R, dn, s, e0, e1)
                              : launch_gemm(GEMM_DOWN, c->bf16, rg, row_tiles, dn, s, e0, e1));
    }
    if (!sh.tail) return CLLM_OK;

    ScanParams sp{};
    sp.ctl = c->ctl;
    sp.tab = c->tab;
    sp.rows = c->rows;
    sp.cap = c->cap;
    sp.pmax = c->pmax;
    sp.pidx = c->pidx;
    sp.n_wg = c->n_wg_lm;
    sp.out = out_dev;
    sp.stream = stream_dev;
    sp.out_stride = c->opts.max_new;
    sp.stream_stride = c->stream_cap;
    sp.plan_inline = sh.nseq == 1;
    sp.mlog = out_dev ? c->mlog_dev : nullptr;
    sp.trace = (out_dev && c->trace_on) ? c->trace_dev : nullptr;
    sp.trace_cap = c->opts.max_new;
    if (sh.with_lm) {
        GemmParams lm = base;
        lm.W = c->w_lm;
        lm.Ks = c->ks_d;
        lm.cols = c->n_wg_lm * 16 * kLmTiles;
        lm.A = c->An;
        lm.lda = c->d;
        lm.pmax = c->pmax;
        lm.pidx = c->pidx;
        lm.dbg = c->dbg_on ? c->dbg : nullptr;
        int lm_tiles = row_tiles;
        if (sh.lm_mask && tiled) {  // one launch per tile that holds a prompt's last row
            for (int t = 0; t < row_tiles; ++t) {
                if (!((sh.lm_mask >> t) & 1)) continue;
                lm.rt0 = t;
                timing_events(c, CLLM_KT_LM_HEAD, rg, &e0, &e1);
                HIPCHK(c, launch_gemm(GEMM_LM, c->bf16, rg, 1, lm, s, e0, e1));
            }
        } else {
            if (sh.lm_rt0 >= 0 && tiled) {
                lm.rt0 = sh.lm_rt0;
                lm_tiles = 1;
            }
            timing_events(c, CLLM_KT_LM_HEAD, rg, &e0, &e1);
            HIPCHK(c, launch_gemm(GEMM_LM, c->bf16, rg, lm_tiles, lm, s, e0, e1));
        }
        sp.advance_only = 0;
        sp.advance_mask = sh.adv_mask;
    } else {
        sp.advance_only = 1;
    }
    timing_events(c, CLLM_KT_SCAN, rg, &e0, &e1);
    HIPCHK(c, launch_scan(sh.nseq, sp, s, e0, e1));
    if (!sp.plan_inline) HIPCHK(c, launch_plan(PlanParams{c->ctl, c->tab, c->rows, c->cap}, s));
    return CLLM_OK;
}

// Host edits for nseq batch entries: slot seq[b] gets mode and block size m[b]; its tokens are
// copied from host zs + b * zstride (packed: entry after entry). Entries with their bit set in
// reset_mask (a prompt's first prefill chunk) restart at L = 0.
cllm_status setup(cllm_ctx *c, int mode, int nseq, const int32_t *seq, const int32_t *m, const int32_t *zs, int zstride,
                  uint64_t reset_mask, bool packed = false) {
    SetupParams sp{};
    sp.ctl = c->ctl;
    sp.tab = c->tab;
    sp.rows = c->rows;
    sp.zin = c->zin;
    sp.zstride = zstride;
    sp.packed = packed ? 1 : 0;
    sp.nseq = nseq;
    sp.mode = mode;
    sp.reset_mask = reset_mask;
    size_t ntok = 0, npacked = 0;
    for (int b = 0; b < nseq; ++b) {
        sp.seq[b] = seq[b];
        sp.m[b] = m[b];
        npacked += m[b];
        ntok = std::max(ntok, packed ? npacked : (size_t)b * zstride + m[b]);
    }
    if (ntok > (size_t)c->zin_cap) return fail(c, CLLM_ERR_CAPACITY, "token staging too small");
    if (ntok) HIPCHK(c, hipMemcpyAsync(c->zin, zs, ntok * 4, hipMemcpyHostToDevice, c->stream));
    HIPCHK(c, launch_setup(sp, c->stream));
    return CLLM_OK;
}

// A NaN logit in slot seq (see Slot::dirty).
cllm_status numeric_fail(cllm_ctx *c, int seq, const char *where) {
    c->slot[seq].dirty = true;
    return fail(c, CLLM_ERR_NUMERIC, "NaN logit%s (slot %d)", where, seq);
}

// Zero the key and value caches of a slot that reported a NaN logit, before its next prefill.
cllm_status clear_if_dirty(cllm_ctx *c, int seq) {
    if (!c->slot[seq].dirty) return CLLM_OK;
    const size_t bytes = c->kv_seq * c->elem;
    HIPCHK(c, hipMemsetAsync(static_cast<uint8_t *>(c->kc) + (size_t)seq * bytes, 0, bytes, c->stream));
    HIPCHK(c, hipMemsetAsync(static_cast<uint8_t *>(c->vt) + (size_t)seq * bytes, 0, bytes, c->stream));
    c->slot[seq].dirty = false;
    return CLLM_OK;
}

// Read the control blocks of every slot (h: max_batch entries).
cllm_status read_ctl(cllm_ctx *c, Ctl *h) {
    HIPCHK(c, hipMemcpyAsync(h, c->ctl, sizeof(Ctl) * c->max_batch, hipMemcpyDeviceToHost, c->stream));
    HIPCHK(c, hipStreamSynchronize(c->stream));
    if (c->kt_class >= 0) timing_collect(c);
    return CLLM_OK;
}

cllm_status check_ids(cllm_ctx *c, const int32_t *ids, int n) {
    for (int i = 0; i < n; ++i)
        if (ids[i] < 0 || ids[i] >= c->V) return fail(c, CLLM_ERR_ARG, "token id %d at index %d out of range", ids[i], i);
    return CLLM_OK;
}

// Prefill of one slot in chunks of the row capacity; the LM head runs on the last chunk's last
// row tile only.
cllm_status prefill_impl(cllm_ctx *c, int seq, const int32_t *prompt, int len) {
    c->slot[seq].prefilled = false;
    if (cllm_status st = clear_if_dirty(c, seq)) return st;
    c->in_prefill = true;
    struct Flag {  // cleared on every return
        bool &f;
        ~Flag() { f = false; }
    } flag{c->in_prefill};
    const int chunk = c->pchunk;
    const int nchunks = ceil_div(len, chunk);
    for (int k = 0; k < nchunks; ++k) {
        const int start = k * chunk;
        const int rows = std::min(chunk, len - start);
        cllm_status st = setup(c, MODE_PREFILL, 1, &seq, &rows, prompt + start, chunk, k == 0 ? 1 : 0);
        if (st) return st;
        const bool last = k == nchunks - 1;
        IterShape sh{rows, 1, rows, std::min(c->nch, ceil_div(start + rows, kAttnChunk)), last,
                     last ? (rows - 1) / kMaxRows : -1};
        sh.prompt = true;
        st = enqueue_iteration(c, sh, nullptr, nullptr);
        if (st) return st;
    }
    return CLLM_OK;
}

// Prefill of B prompts packed into passes of up to the prefill chunk: each pass takes the
// remaining rows of the prompts in order (a prompt may span passes), so short prompts share a
// pass instead of each streaming the weights on its own. The LM head runs on the 64-row tiles
// that hold a prompt's last row; entries whose rows do not end their prompt only advance. Every
// prompt row takes the prompt GEMM and the chunk-parallel attention at absolute positions, so the
// caches and first tokens are those of one prefill per prompt.
static_assert(kMaxPrefillRows <= 64 * kMaxRows && kMaxSeqs <= 64, "one mask bit per row tile and per entry");
cllm_status prefill_packed_impl(cllm_ctx *c, int B, const int32_t *seq_ids, const int32_t *prompts,
                                const size_t *off, const int32_t *lens) {
    for (int b = 0; b < B; ++b) {
        c->slot[seq_ids[b]].prefilled = false;
        if (cllm_status st = clear_if_dirty(c, seq_ids[b])) return st;
    }
    c->in_prefill = true;
    struct Flag {  // cleared on every return
        bool &f;
        ~Flag() { f = false; }
    } flag{c->in_prefill};
    const int chunk = c->pchunk;
    std::vector<int> done(B, 0);  // prompt rows already prefilled
    std::vector<int32_t> seq, m;
    int b = 0;
    while (b < B) {
        seq.clear();
        m.clear();
        // the pass's tokens are one contiguous run of the concatenated prompts (the caller's
        // buffer, valid for the whole call)
        const int32_t *zs = prompts + off[b] + done[b];
        uint64_t reset = 0, adv = 0, lm = 0;
        int R = 0, maxm = 0, nch = 1;
        while (b < B && R < chunk && (int)seq.size() < kMaxSeqs) {
            const int e = (int)seq.size(), take = std::min(lens[b] - done[b], chunk - R);
            seq.push_back(seq_ids[b]);
            m.push_back(take);
            if (done[b] == 0) reset |= 1ull << e;
            done[b] += take;
            nch = std::max(nch, ceil_div(done[b], kAttnChunk));
            maxm = std::max(maxm, take);
            R += take;
            if (done[b] == lens[b]) {
                lm |= 1ull << ((R - 1) / kMaxRows);
                ++b;
            } else {
                adv |= 1ull << e;
            }
        }
        const int ne = (int)seq.size();
        cllm_status st = setup(c, MODE_PREFILL, ne, seq.data(), m.data(), zs, 0, reset, true);
        if (st) return st;
        IterShape sh{R, ne, maxm, std::min(c->nch, nch), lm != 0, -1};
        sh.prompt = true;
        sh.lm_mask = R > kMaxRows ? lm : 0;
        sh.adv_mask = adv;
        st = enqueue_iteration(c, sh, nullptr, nullptr);
        if (st) return st;
    }
    return CLLM_OK;
}

cllm_status check_ctx(cllm_ctx *c) {
    if (c->dead) return fail(c, CLLM_ERR_DEVICE, "context unusable after a device error: %s", c->err.c_str());
    return CLLM_OK;
}

cllm_status check_seq(cllm_ctx *c, int32_t seq) {
    if (seq < 0 || seq >= c->max_batch) return fail(c, CLLM_ERR_ARG, "seq %d outside [0, %d)", seq, c->max_batch);
    return CLLM_OK;
}

// One batched iteration over B entries (host-driven step): validate, run, read back.
cllm_status step_batch_impl(cllm_ctx *c, int32_t B, const int32_t *seq_ids, const int32_t *blocks_in, int32_t zstride,
                            const int32_t *m, int32_t *blocks_out, int32_t ostride, int32_t *accepted) {
    if (B < 1 || B > c->max_batch) return fail(c, CLLM_ERR_ARG, "B=%d outside [1, max_batch]", B);
    if (!seq_ids || !blocks_in || !m || !blocks_out || !accepted) return fail(c, CLLM_ERR_ARG, "NULL pointer");
    std::vector<char> seen(c->max_batch, 0);
    int R = 0, maxm = 0, nch = 1;
    cllm_status s;
    for (int b = 0; b < B; ++b) {
        const int q = seq_ids[b];
        if ((s = check_seq(c, q))) return s;
        if (seen[q]) return fail(c, CLLM_ERR_ARG, "slot %d appears twice", q);
        seen[q] = 1;
        if (m[b] < 1 || m[b] > c->opts.max_block) return fail(c, CLLM_ERR_ARG, "m=%d outside [1, max_block]", m[b]);
        if (!c->slot[q].prefilled) return fail(c, CLLM_ERR_STATE, "jacobi step before prefill (slot %d)", q);
        const int32_t *z = blocks_in + (size_t)b * zstride;
        if ((s = check_ids(c, z, m[b]))) return s;
        if (z[0] != c->slot[q].pending)
            return fail(c, CLLM_ERR_STATE, "block_in[0]=%d is not the pending token %d (slot %d)", z[0],
                        c->slot[q].pending, q);
        if (c->slot[q].L + m[b] > c->opts.max_ctx) return fail(c, CLLM_ERR_CAPACITY, "L + m exceeds max_ctx");
        R += m[b];
        maxm = std::max(maxm, m[b]);
        nch = std::max(nch, ceil_div(c->slot[q].L + m[b], kAttnChunk));
    }
    if ((s = setup(c, MODE_STEP, B, seq_ids, m, blocks_in, zstride, 0))) return s;
    const IterShape sh{R, B, maxm, nch, true, -1};
    if ((s = enqueue_iteration(c, sh, nullptr, nullptr))) return s;
    std::vector<Ctl> h(c->max_batch);
    if ((s = read_ctl(c, h.data()))) return s;
    for (int b = 0; b < B; ++b)
        if (h[seq_ids[b]].err) return numeric_fail(c, seq_ids[b], "");
    if (c->dbg_on && c->dbg_host)
        HIPCHK(c, hipMemcpy(c->dbg_host, c->dbg, (size_t)std::min(R, c->dbg_rows) * c->V * 4, hipMemcpyDeviceToHost));
    for (int b = 0; b < B; ++b) {
        const Ctl &ct = h[seq_ids[b]];
        for (int i = 0; i < m[b]; ++i) blocks_out[(size_t)b * ostride + i] = ct.pred[i];
        accepted[b] = ct.a_last;
        c->slot[seq_ids[b]].L = ct.L;
        c->slot[seq_ids[b]].pending = ct.pending;
    }
    return CLLM_OK;
}

// Prefill B prompts, then decode max_new tokens each in one device-resident loop.
cllm_status decode_batch_impl(cllm_ctx *c, int32_t B, const int32_t *seq_ids, const int32_t *prompts,
                              const int32_t *lens, int32_t n, int32_t max_new, const cllm_guess_spec *guesses,
                              int32_t *out_tokens, cllm_decode_stats *stats) {
    if (B < 1 || B > c->max_batch) return fail(c, CLLM_ERR_ARG, "B=%d outside [1, max_batch]", B);
    if (!seq_ids || !prompts || !lens || !out_tokens) return fail(c, CLLM_ERR_ARG, "NULL pointer");
    if (n < 1 || n > c->opts.max_block) return fail(c, CLLM_ERR_ARG, "n=%d outside [1, max_block]", n);
    if (max_new < 1) return fail(c, CLLM_ERR_ARG, "max_new must be >= 1");
    if (max_new > c->opts.max_new) return fail(c, CLLM_ERR_CAPACITY, "max_new exceeds the context's max_new");
    cllm_status s;
    std::vector<char> seen(c->max_batch, 0);
    std::vector<cllm_guess_spec> gs(B);
    std::vector<size_t> off(B + 1, 0);
    int maxlen = 0;
    for (int b = 0; b < B; ++b) {
        const int q = seq_ids[b];
        if ((s = check_seq(c, q))) return s;
        if (seen[q]) return fail(c, CLLM_ERR_ARG, "slot %d appears twice", q);
        seen[q] = 1;
        if (lens[b] < 1) return fail(c, CLLM_ERR_ARG, "bad prompt length");
        if (lens[b] + max_new + n > c->opts.max_ctx)
            return fail(c, CLLM_ERR_CAPACITY, "len + max_new + n exceeds max_ctx");
        off[b + 1] = off[b] + lens[b];
        maxlen = std::max(maxlen, lens[b]);
        if (guesses) gs[b] = guesses[b];
        const cllm_guess_spec &g = gs[b];
        if (g.policy < 0 || g.policy > 2 || g.block_policy < 0 || g.block_policy > 1)
            return fail(c, CLLM_ERR_ARG, "bad guess policy");
        if (g.policy != CLLM_GUESS_UNIFORM) {
            if (!g.stream || g.stream_len < max_new) return fail(c, CLLM_ERR_ARG, "guess stream shorter than max_new");
            if (g.thr53 > (1ull << 53)) return fail(c, CLLM_ERR_ARG, "thr53 above 2^53");
        }
    }
    for (int b = 0; b < B; ++b) {
        if ((s = check_ids(c, prompts + off[b], lens[b]))) return s;
        if (gs[b].policy != CLLM_GUESS_UNIFORM && (s = check_ids(c, gs[b].stream, max_new))) return s;
    }

    hipEvent_t ev[3];
    for (auto &e : ev) HIPCHK(c, hipEventCreate(&e));
    struct EvGuard {
        hipEvent_t *e;
        ~EvGuard() {
            for (int i = 0; i < 3; ++i) (void)hipEventDestroy(e[i]);
        }
    } guard{ev};

    bool any_stream = false;
    for (int b = 0; b < B; ++b)
        if (gs[b].policy != CLLM_GUESS_UNIFORM) {
            any_stream = true;
            HIPCHK(c, hipMemcpyAsync(c->stream_dev + (size_t)seq_ids[b] * c->stream_cap, gs[b].stream,
                                     (size_t)max_new * 4, hipMemcpyHostToDevice, c->stream));
        }
    HIPCHK(c, hipEventRecord(ev[0], c->stream));
    if ((s = prefill_packed_impl(c, B, seq_ids, prompts, off.data(), lens))) return s;
    HIPCHK(c, hipEventRecord(ev[1], c->stream));
    // Decode parameters into the control blocks (the prefill left L and pending there).
    std::vector<Ctl> h(c->max_batch);
    if ((s = read_ctl(c, h.data()))) return s;
    for (int b = 0; b < B; ++b) {
        Ctl &ct = h[seq_ids[b]];
        if (ct.err) return numeric_fail(c, seq_ids[b], " in the prefill");
        ct.n = n;
        ct.max_new = max_new;
        ct.policy = gs[b].policy;
        ct.block_policy = gs[b].block_policy;
        ct.seq = seq_ids[b];
        ct.stream_len = gs[b].policy != CLLM_GUESS_UNIFORM ? max_new : 0;
        ct.vocab = c->V;
        ct.seed = gs[b].seed;
        ct.thr53 = gs[b].thr53;
    }
    HIPCHK(c, hipMemcpyAsync(c->ctl, h.data(), sizeof(Ctl) * c->max_batch, hipMemcpyHostToDevice, c->stream));
    // the batch entries into the row table, then the first blocks and their rows
    std::vector<int32_t> zero_m(B, 0);
    if ((s = setup(c, MODE_DECODE, B, seq_ids, zero_m.data(), nullptr, 0, 0))) return s;
    ScanParams sp{};
    sp.ctl = c->ctl;
    sp.tab = c->tab;
    sp.stream = any_stream ? c->stream_dev : nullptr;
    sp.stream_stride = c->stream_cap;
    HIPCHK(c, launch_decode_init(B, sp, c->stream));
    HIPCHK(c, launch_plan(PlanParams{c->ctl, c->tab, c->rows, c->cap}, c->stream));
    IterShape sh{B * n, B, n, std::min(c->nch, ceil_div(maxlen + max_new + n, kAttnChunk)), true, -1};
    if (!c->ctl_snap) {
        void *hp = nullptr;
        HIPCHK(c, hipHostMalloc(&hp, sizeof(Ctl) * c->max_batch, hipHostMallocDefault));
        c->ctl_snap = static_cast<Ctl *>(hp);
        HIPCHK(c, hipEventCreateWithFlags(&c->snap_ev, hipEventDisableTiming));
    }
    // Device-resident loop: every launch reads its rows from the row table. The host only
    // queues iterations: as many as are certainly needed by the sequence with the most tokens
    // left (each iteration fixes at most n tokens of a sequence). The control blocks are copied
    // out before a round's last iteration and read while it runs, so the next round is queued
    // before the GPU runs dry; that iteration may still fix up to n tokens of each sequence
    // (lag), so the next round is shorter by one. When nothing is certainly needed beyond the
    // iterations in flight, the host waits for them and looks again.
    int64_t queued = 0;
    size_t nev = 0;  // iteration events recorded
    int lag = 0;     // iterations queued after the state in h was taken
    auto check_err = [&]() -> cllm_status {
        for (int b = 0; b < B; ++b)
            if (h[seq_ids[b]].err) return numeric_fail(c, seq_ids[b], "");
        return CLLM_OK;
    };
    while (true) {
        int need = 0;
        for (int b = 0; b < B; ++b) {
            const Ctl &ct = h[seq_ids[b]];
            const int left = ct.done ? 0 : max_new - (queued ? ct.e : 0);
            need = std::max(need, ceil_div(left, n));
        }
        need -= lag;
        if (need <= 0) {
            if (lag == 0) break;
            if ((s = read_ctl(c, h.data()))) return s;  // the iterations in flight have finished
            lag = 0;
            if ((s = check_err())) return s;
            continue;
        }
        // Launch shape of this round: the blocks of the sequences still running (a finished
        // sequence's block is empty in the row table, and a row's values do not depend on the
        // launch shape), so the products of the last rounds launch for fewer row tiles.
        int active = 0;
        for (int b = 0; b < B; ++b) active += h[seq_ids[b]].done ? 0 : 1;
        sh.R = std::max(active, 1) * n;
        for (int i = 0; i < need; ++i) {
            if (i == need - 1) {  // the state before the round's last iteration
                HIPCHK(c, hipMemcpyAsync(c->ctl_snap, c->ctl, sizeof(Ctl) * c->max_batch, hipMemcpyDeviceToHost,
                                         c->stream));
                HIPCHK(c, hipEventRecord(c->snap_ev, c->stream));
            }
            if ((s = enqueue_iteration(c, sh, c->out_dev, any_stream ? c->stream_dev : nullptr))) return s;
            if (nev == c->it_ev.size()) {
                hipEvent_t e;
                HIPCHK(c, hipEventCreate(&e));
                c->it_ev.push_back(e);
            }
            HIPCHK(c, hipEventRecord(c->it_ev[nev++], c->stream));
        }
        queued += need;
        HIPCHK(c, hipEventRecord(ev[2], c->stream));
        HIPCHK(c, hipEventSynchronize(c->snap_ev));
        std::copy(c->ctl_snap, c->ctl_snap + c->max_batch, h.begin());
        lag = 1;
        if ((s = check_err())) return s;
        if (queued > (int64_t)max_new + 1) return fail(c, CLLM_ERR_STATE, "decode did not finish");
    }
    float pre_ms = 0.f, dec_ms = 0.f;
    (void)hipEventElapsedTime(&pre_ms, ev[0], ev[1]);
    (void)hipEventElapsedTime(&dec_ms, ev[1], ev[2]);
    // Per-iteration device times over the iterations that ran (the queue may hold a few past the
    // end, which exit at once) and, with one sequence, the block size of each.
    int64_t real = 0;
    for (int b = 0; b < B; ++b) real = std::max<int64_t>(real, h[seq_ids[b]].steps);
    real = std::min<int64_t>(real, (int64_t)nev);
    std::vector<double> it_ms, full_ms;
    std::vector<int32_t> mlog(B == 1 ? (size_t)real : 0);
    if (B == 1 && real > 0)
        HIPCHK(c, hipMemcpy(mlog.data(), c->mlog_dev + (size_t)seq_ids[0] * c->opts.max_new, (size_t)real * 4,
                            hipMemcpyDeviceToHost));
    for (int64_t i = 0; i < real; ++i) {
        float ms = 0.f;
        if (hipEventElapsedTime(&ms, i ? c->it_ev[i - 1] : ev[1], c->it_ev[i]) != hipSuccess) continue;
        it_ms.push_back(ms);
        if (B == 1 && mlog[i] == n) full_ms.push_back(ms);
    }
    auto pct = [](std::vector<double> v, double q) {
        if (v.empty()) return 0.0;
        std::sort(v.begin(), v.end());
        return v[(size_t)(q * (double)(v.size() - 1) + 0.5)];
    };
    const double p10 = pct(it_ms, 0.1), p50 = pct(it_ms, 0.5), p90 = pct(it_ms, 0.9);
    const double full50 = B == 1 ? pct(full_ms, 0.5) : p50;
    const double full10 = B == 1 ? pct(full_ms, 0.1) : p10, full90 = B == 1 ? pct(full_ms, 0.9) : p90;
    for (int b = 0; b < B; ++b) {
        const int q = seq_ids[b];
        HIPCHK(c, hipMemcpy(out_tokens + (size_t)b * max_new, c->out_dev + (size_t)q * c->opts.max_new,
                            (size_t)max_new * 4, hipMemcpyDeviceToHost));
        const Ctl &ct = h[q];
        if (stats) {
            cllm_decode_stats &st = stats[b];
            memset(&st, 0, sizeof(st));
            st.steps = ct.steps;
            st.rows = ct.rows;
            st.blocks = ct.blocks;
            st.tokens = ct.e;
            for (int i = 0; i <= kMaxBlock; ++i) st.accept_hist[i] = ct.hist[i];
            st.prefill_ms = pre_ms;
            st.decode_ms = dec_ms;
            st.iter_ms_p10 = p10;
            st.iter_ms_p50 = p50;
            st.iter_ms_p90 = p90;
            st.iter_ms_full_p50 = full50;
            st.iter_ms_full_p10 = full10;
            st.iter_ms_full_p90 = full90;
        }
        c->slot[q].prefilled = true;
        c->slot[q].L = ct.L;
        c->slot[q].pending = ct.pending;
        c->slot[q].trace_n = c->trace_on ? std::min<int64_t>(ct.steps, c->opts.max_new) : 0;
    }
    return CLLM_OK;
}

}  // namespace

// ------------------------------------------------------------------------------------------
// Fixed scratch of cllm_hidden_rows_noalloc: the staging buffer of the LM-head input rows of one
// call (m x d_model floats, at most kMaxBlock x 8192), a file-scope device array instead of an
// allocation. Every GPU the library runs on holds its own copy until the process ends; its
// address on a device is taken once, at the first context creation on that device (the array's
// name is not a device address in host code). Calls on one GPU share it.
// ------------------------------------------------------------------------------------------
constexpr size_t kNoAllocFloats = (size_t)kMaxBlock * 8192;
static __device__ __align__(256) float scratch[kNoAllocFloats];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
float *g_scratch_dev[kMaxDevices] = {};  // scratch's device address per device ordinal

// With device `dev` current: look up scratch's address on it (once per device).
cllm_status scratch_setup(cllm_ctx *c, int dev) {
    if (dev < 0 || dev >= kMaxDevices) return fail(c, CLLM_ERR_ARG, "device ordinal %d beyond %d", dev, kMaxDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (g_scratch_dev[dev]) return CLLM_OK;
    void *p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
        return fail(c, CLLM_ERR_DEVICE, "hipGetSymbolAddress(scratch) failed: %s", hipGetErrorString(e));
    g_scratch_dev[dev] = static_cast<float *>(p);
    return CLLM_OK;
}

float *scratch_of(int dev) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    return dev >= 0 && dev < kMaxDevices ? g_scratch_dev[dev] : nullptr;
}
}  // namespace

// ------------------------------------------------------------------------------------------
// C ABI
// ------------------------------------------------------------------------------------------
namespace {
// Grow a loss-head workspace buffer (contents are not kept).
template <class T>
cllm_status loss_buf(cllm_ctx *c, T **p, size_t *have, size_t need) {
    if (*have >= need && *p) return CLLM_OK;
    if (*p) {
        (void)hipFree(*p);
        c->allocs.erase(std::find(c->allocs.begin(), c->allocs.end(), (void *)*p));
        *p = nullptr;
    }
    *have = 0;
    cllm_status s = dalloc_t(c, p, need);
    if (s == CLLM_OK) *have = need;
    return s;
}

bool loss_args_ok(const float *teacher, const float *student, int32_t n_pairs, const float *ar_rows,
                  const int32_t *ar_targets, int32_t n_ar, float omega, const float *row_kl, const float *row_nll,
                  const float *d_student, const float *d_ar) {
    return n_pairs >= 0 && n_ar >= 0 && n_pairs + n_ar >= 1 && n_pairs + n_ar <= 64 &&
           (n_pairs == 0 || (teacher && student && row_kl && d_student)) &&
           (n_ar == 0 || (ar_rows && ar_targets && row_nll && d_ar)) && omega == omega;
}

// Memory a kernel on the context's GPU may access: device memory of that GPU, managed memory, or
// pinned host memory (pageable host memory is not known to the runtime and fails the query).
bool device_accessible(cllm_ctx *c, const void *p) {
    hipPointerAttribute_t a{};
    if (hipPointerGetAttributes(&a, p) != hipSuccess) {
        (void)hipGetLastError();
        return false;
    }
    if (a.type == hipMemoryTypeDevice) return a.device == c->opts.device;
    return a.type == hipMemoryTypeManaged || a.type == hipMemoryTypeHost || a.isManaged;
}

// The loss head on device arrays, enqueued on the context's stream: pack the rows into the GEMM
// operand, logits through the LM head, per-row losses and logit gradients D, D (and H) packed as
// MFMA operands, dH = D W through the transposed LM head (K split over workgroups, partials
// summed in split order), dW = D^T H (if d_weight) and the total (if loss). The workspace grows
// on demand (hipMalloc); the transposed LM head is built on the first call after the weights
// are set.
cllm_status loss_head_enqueue(cllm_ctx *c, const float *T, const float *S, int P, const float *Ar, const int32_t *tg,
                              int A, float omega, float *kl, float *nll, float *dS, float *dA, float *dW,
                              double *loss) {
    const int R = 2 * P + A, Rg = P + A, d = c->d, V = c->V;
    if (R > 2 * kMaxRows) return fail(c, CLLM_ERR_ARG, "loss head: %d GEMM rows exceed %d", R, 2 * kMaxRows);
    const int Vp = c->n_wg_lm * 16 * kLmTiles;
    const int cap = round_up(R, kMaxRows);
    const int nch = ceil_div(Vp, kLossChunk);
    const int rpad = round_up(Rg, 32);
    const int kstep = c->bf16 ? 32 : 16;  // MFMA k-step (elements)
    // dH splits: about 512 workgroups over the columns of d and the vocabulary's k-steps
    const int ks_v = Vp / kstep, n_wg_dh = ceil_div(d, 16 * kLmTiles);
    const int kc = ceil_div(ks_v, std::max(1, std::min(ks_v, ceil_div(512, n_wg_dh))));
    const int nsplit = ceil_div(ks_v, kc);
    auto &w = c->loss;
    cllm_status s;
    if ((s = loss_buf(c, &w.A, &w.a, (size_t)cap * d * 4)) || (s = loss_buf(c, &w.Z, &w.z, (size_t)R * Vp)) ||
        (s = loss_buf(c, &w.D, &w.dd, (size_t)Rg * Vp)) || (s = loss_buf(c, &w.stats, &w.st, (size_t)Rg * nch * 5)) ||
        (s = loss_buf(c, &w.Dact, &w.da, (size_t)kMaxRows * Vp * 4)) ||
        (s = loss_buf(c, &w.part_p, &w.part, (size_t)nsplit * Rg * d)))
        return s;
    if (c->bf16 && ((s = loss_buf(c, &w.DT, &w.dt, (size_t)2 * Vp * rpad)) ||
                    (s = loss_buf(c, &w.HT, &w.ht, (size_t)2 * d * rpad))))
        return s;
    hipStream_t st = c->stream;
    if (!w.tabs) {  // once per context: every row count's table (rows of one block, no positions)
        if ((s = dalloc_t(c, &w.tabs, 2 * kMaxRows))) return s;
        std::vector<RowTab> th(2 * kMaxRows);
        for (int i = 0; i < 2 * kMaxRows; ++i) {
            th[i].R = i + 1;
            th[i].nseq = 1;
        }
        HIPCHK(c, hipMemcpyAsync(w.tabs, th.data(), th.size() * sizeof(RowTab), hipMemcpyHostToDevice, st));
        HIPCHK(c, hipStreamSynchronize(st));
    }
    if (!w.wt_ok) {  // the LM head as the weight operand of dH = D W
        if (!w.WT && (s = dalloc_t(c, &w.WT, (size_t)Vp * d * c->elem))) return s;
        HIPCHK(c, launch_transpose_lm(c->bf16, c->w_lm, Vp, d, w.WT, st));
        w.wt_ok = true;
    }
    hipEvent_t e0, e1;
    // logits Z = H W^T over the packed LM head (no RMSNorm row factor: the rows are the head's input)
    timing_events(c, CLLM_KT_LOSS_LOGITS, 0, &e0, &e1);
    HIPCHK(c, launch_pack_rows(c->bf16, T, S, P, Ar, A, d, cap, w.A, st, e0));
    GemmParams g{};
    g.W = c->w_lm;
    g.Ks = c->ks_d;
    g.cols = Vp;
    g.A = w.A;
    g.lda = d;
    g.rr = RowsRef{w.tabs + (R - 1), nullptr, cap};
    g.V = V;
    g.Zout = w.Z;
    g.ldz = Vp;
    // one launch per 64-row tile (each streams the weights once; measured faster than one launch
    // of two row tiles sharing them), each sized to its rows
    const int row_tiles = ceil_div(R, kMaxRows);
    for (int t = 0; t < row_tiles; ++t) {
        const int rg = rows_to_rg(std::min(kMaxRows, R - t * kMaxRows));
        g.rt0 = t * kMaxRows / (16 * rg);  // in units of the launch's 16 * rg rows
        HIPCHK(c, launch_gemm(GEMM_LOGITS, c->bf16, rg, 1, g, st, nullptr, t == row_tiles - 1 ? e1 : nullptr));
    }
    // per-row losses, D, and D (and H) as MFMA operands
    LossParams lp{w.Z, tg, P, A, V, Vp, omega, kl, nll, w.D};
    timing_events(c, CLLM_KT_LOSS_ROWS, 0, &e0, &e1);
    HIPCHK(c, launch_loss_rows(lp, w.stats, st, e0, nullptr));
    HIPCHK(c, launch_loss_pack(c->bf16, w.D, Rg, Vp, Vp, kMaxRows, w.Dact, rpad, w.DT, S, P, Ar, d, w.HT, st, e1));
    // dH = D W: the streaming GEMM over the transposed LM head, K (the vocabulary) split nsplit ways
    GemmParams h{};
    h.W = w.WT;
    h.Ks = ks_v;
    h.cols = d;
    h.A = w.Dact;
    h.lda = Vp;
    h.rr = RowsRef{w.tabs + (Rg - 1), nullptr, kMaxRows};
    h.V = d;
    h.Zout = w.part_p;
    h.ldz = d;
    h.kc = kc;
    h.zstride = (size_t)Rg * d;
    timing_events(c, CLLM_KT_LOSS_DH, 0, &e0, &e1);
    HIPCHK(c, launch_gemm(GEMM_LOGITS, c->bf16, rows_to_rg(Rg), 1, h, st, e0, nullptr));
    HIPCHK(c, launch_loss_dh_sum(w.part_p, nsplit, Rg, d, P, dS, dA, st, e1));
    if (dW) {
        timing_events(c, CLLM_KT_LOSS_DW, 0, &e0, &e1);
        HIPCHK(c, launch_loss_dw(c->bf16, w.DT, w.HT, Vp, rpad, w.D, Rg, Vp, S, P, Ar, d, V, dW, st, e0, e1));
    }
    if (loss) HIPCHK(c, launch_loss_total(kl, P, nll, A, omega, loss, st));
    return CLLM_OK;
}

// SplitMix64 output function (Steele, Lea and Flood, OOPSLA 2014): the host side of the weight
// generator's keys and the collection's augmentation draws.
uint64_t splitmix64(uint64_t x) {
    x += 0x9E3779B97F4A7C15ull;
    x = (x ^ (x >> 30)) * 0xBF58476D1CE4E5B9ull;
    x = (x ^ (x >> 27)) * 0x94D049BB133111EBull;
    return x ^ (x >> 31);
}

// Where the weight tensors come from: host arrays in the order of cllm_model_set_weights, or
// (host == NULL) the seeded generator, drawn on the device.
struct WeightSource {
    const void *const *host;
    uint64_t seed;
};

// Generator stream of tensor idx (the order of cllm_model_set_weights) and whether it is a norm
// gain (1.0) rather than a N(0, 0.02) matrix.
void tensor_stream(int NL, int idx, uint64_t *stream, bool *gain) {
    if (idx == 0) {
        *stream = 1, *gain = false;
    } else if (idx == 1 + 9 * NL) {
        *stream = 2, *gain = true;
    } else if (idx == 2 + 9 * NL) {
        *stream = 3, *gain = false;
    } else {
        const int l = (idx - 1) / 9, t = (idx - 1) % 9;
        *stream = 1000ull * (uint64_t)(l + 1) + (uint64_t)t;
        *gain = t == 0 || t == 5;
    }
}

// Writes tensor idx (elems elements: float for gains, the model's element type otherwise) to
// device memory dst, from the host array or from the generator.
cllm_status put_tensor(cllm_ctx *c, const WeightSource &src, int idx, void *dst, size_t elems) {
    uint64_t stream;
    bool gain;
    tensor_stream(c->NL, idx, &stream, &gain);
    if (src.host) {
        HIPCHK(c, hipMemcpyAsync(dst, src.host[idx], elems * (gain ? 4 : c->elem), hipMemcpyHostToDevice, c->stream));
        return CLLM_OK;
    }
    const uint64_t key = splitmix64(splitmix64(src.seed) ^ stream);
    HIPCHK(c, launch_fill_weights(gain ? 2 : (c->bf16 ? 1 : 0), key, kWeightStd, elems, dst, c->stream));
    return CLLM_OK;
}

// Every weight of the model: copied or drawn into place (embedding, norm gains) or into a staging
// buffer and repacked into the streaming layout (the products' matrices).
cllm_status load_weights(cllm_ctx *c, const WeightSource &src) {
    c->loss.wt_ok = false;  // the loss head's transposed LM head is rebuilt on its next call
    const int d = c->d, F = c->F, V = c->V;
    const size_t E = c->elem;
    size_t stage_elems = std::max({(size_t)3 * d * d, (size_t)2 * F * d, (size_t)V * d});
    uint8_t *staging = nullptr;
    int32_t *perm_dev = nullptr;
    if (hipMalloc(reinterpret_cast<void **>(&staging), stage_elems * E) != hipSuccess) {
        (void)hipGetLastError();
        return fail(c, CLLM_ERR_OOM, "staging allocation failed");
    }
    const size_t perm_max = std::max({(size_t)3 * d, (size_t)2 * c->Fp, (size_t)round_up(V, 16 * kLmTiles)});
    if (hipMalloc(reinterpret_cast<void **>(&perm_dev), perm_max * 4) != hipSuccess) {
        (void)hipGetLastError();
        (void)hipFree(staging);
        return fail(c, CLLM_ERR_OOM, "staging allocation failed");
    }
    cllm_status s = CLLM_OK;
    const std::vector<int32_t> pq = qkv_perm(c), pgu = gate_up_perm(c), pd = plain_perm(d, d),
                               plm = plain_perm(round_up(V, 16 * kLmTiles), V);
    c->streamed_bytes = 0;
    const size_t dd = (size_t)d * d, fd = (size_t)F * d;
    do {
        if ((s = put_tensor(c, src, 0, c->embed, (size_t)V * d))) break;
        for (int l = 0; l < c->NL && !s; ++l) {
            const int t = 1 + 9 * l;
            if ((s = put_tensor(c, src, t, c->g_attn[l], d))) break;
            for (int k = 0; k < 3 && !s; ++k) s = put_tensor(c, src, t + 1 + k, staging + k * dd * E, dd);  // [q; k; v]
            if (s || (s = pack_staged(c, d, c->ks_d, pq, &c->w_qkv[l], staging, perm_dev))) break;
            if ((s = put_tensor(c, src, t + 4, staging, dd)) || (s = pack_staged(c, d, c->ks_d, pd, &c->w_o[l], staging, perm_dev)))
                break;
            if ((s = put_tensor(c, src, t + 5, c->g_ffn[l], d))) break;
            if ((s = put_tensor(c, src, t + 6, staging, fd)) || (s = put_tensor(c, src, t + 7, staging + fd * E, fd)) ||
                (s = pack_staged(c, d, c->ks_d, pgu, &c->w_gu[l], staging, perm_dev)))
                break;
            if ((s = put_tensor(c, src, t + 8, staging, fd)) || (s = pack_staged(c, F, c->ks_f, pd, &c->w_d[l], staging, perm_dev)))
                break;
        }
        if (s) break;
        if ((s = put_tensor(c, src, 1 + 9 * c->NL, c->g_final, d))) break;
        if ((s = put_tensor(c, src, 2 + 9 * c->NL, staging, (size_t)V * d)) ||
            (s = pack_staged(c, d, c->ks_d, plm, &c->w_lm, staging, perm_dev)))
            break;
    } while (0);
    hipError_t e = hipStreamSynchronize(c->stream);
    (void)hipFree(staging);
    (void)hipFree(perm_dev);
    if (s) return s;
    if (e != hipSuccess) return fail(c, CLLM_ERR_DEVICE, "weight upload failed: %s", hipGetErrorString(e));
    for (auto &q : c->slot) q = cllm_ctx::Slot{};
    return CLLM_OK;
}
}  // namespace

extern "C" {

const char *cllm_status_string(cllm_status s) {
    // A C caller may pass any int; in C++ loading an enum object whose value lies outside the
    // enumerators' range is undefined, so the value is read from the object's bytes.
    int32_t v = 0;
    static_assert(sizeof(cllm_status) == sizeof(int32_t), "cllm_status is an int");
    std::memcpy(&v, &s, sizeof v);
    switch (v) {
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
    for (hipEvent_t e : c->it_ev) (void)hipEventDestroy(e);
    if (c->snap_ev) (void)hipEventDestroy(c->snap_ev);
    if (c->ctl_snap) (void)hipHostFree(c->ctl_snap);
    delete c;
}

}  // extern "C"

namespace {

bool config_ok(const cllm_config *cfg, const cllm_runtime_opts *opts) {
    const bool bf16 = cfg->dtype == CLLM_DTYPE_BF16;
    if ((cfg->dtype != CLLM_DTYPE_BF16 && cfg->dtype != CLLM_DTYPE_F32) || cfg->n_layers < 1 || cfg->d_model < 1 ||
        cfg->n_heads < 1 || cfg->n_heads * cfg->head_dim != cfg->d_model ||
        !(cfg->head_dim == 32 || cfg->head_dim == 64 || cfg->head_dim == 128 ||
          (bf16 ? cfg->head_dim == 256 : cfg->head_dim == 16)) ||
        cfg->d_model % 64 != 0 || cfg->d_model > 8192 ||
        cfg->ffn_dim < 1 || cfg->vocab < 2 || !(cfg->rms_eps >= 0.0f) || !(cfg->rope_base > 0.0f))
        return false;
    if (opts->max_block < 1 || opts->max_block > kMaxBlock || opts->max_ctx < 2 ||
        opts->max_ctx > kMaxChunks * kAttnChunk - 2 * kMaxRows || opts->max_new < 1 || opts->max_batch < 0 ||
        opts->max_batch > kMaxSeqs || opts->prefill_chunk < 0 || opts->prefill_chunk > kMaxPrefillRows)
        return false;
    return !(opts->workspace_bytes > 0 && !opts->workspace);
}

// Shape-derived fields of a context (no device calls).
void derive_shape(cllm_ctx *c, const cllm_config *cfg, const cllm_runtime_opts *opts) {
    const bool bf16 = cfg->dtype == CLLM_DTYPE_BF16;
    const int kstep = bf16 ? 32 : 16;
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
    c->n_wg_lm = round_up(c->V, 16 * kLmTiles) / (16 * kLmTiles);
    c->stream = static_cast<hipStream_t>(opts->stream);
    c->max_batch = opts->max_batch > 0 ? opts->max_batch : 1;
    c->opts.max_batch = c->max_batch;
    c->dbg_rows = round_up(std::max(kMaxRows, c->max_batch * opts->max_block), kMaxRows);
    c->pchunk = std::min(round_up(opts->prefill_chunk > 0 ? opts->prefill_chunk : kDefaultPrefillRows, kMaxRows),
                         round_up(opts->max_ctx, kMaxRows));
    c->cap = round_up(std::max(c->dbg_rows, c->pchunk), kPromptRows);  // whole prompt-GEMM row tiles
    c->kv_seq = (size_t)c->NL * c->ctx_alloc * c->d;
}

}  // namespace

extern "C" {

cllm_status cllm_workspace_bytes(const cllm_config *cfg, const cllm_runtime_opts *opts, size_t *bytes) {
    if (!cfg || !opts || !bytes) return CLLM_ERR_ARG;
    *bytes = 0;
    cllm_runtime_opts o = *opts;
    o.workspace = nullptr;
    o.workspace_bytes = 0;
    if (!config_ok(cfg, &o)) return CLLM_ERR_ARG;
    cllm_ctx *c = new (std::nothrow) cllm_ctx;
    if (!c) return CLLM_ERR_OOM;
    derive_shape(c, cfg, &o);
    *bytes = workspace_total(workspace_bufs(c));
    delete c;
    return CLLM_OK;
}

cllm_status cllm_model_create(const cllm_config *cfg, const cllm_runtime_opts *opts, cllm_ctx **out) {
    if (!cfg || !opts || !out) return CLLM_ERR_ARG;
    *out = nullptr;
    if (!config_ok(cfg, opts)) return CLLM_ERR_ARG;
    const int kstep = cfg->dtype == CLLM_DTYPE_BF16 ? 32 : 16;
    int ndev = 0;
    if (hipGetDeviceCount(&ndev) != hipSuccess || opts->device < 0 || opts->device >= ndev) {
        (void)hipGetLastError();
        return CLLM_ERR_DEVICE;
    }
    cllm_ctx *c = new (std::nothrow) cllm_ctx;
    if (!c) return CLLM_ERR_OOM;
    derive_shape(c, cfg, opts);
    c->slot.assign(c->max_batch, cllm_ctx::Slot{});

    auto bail = [&](cllm_status s) {
        cllm_model_free(c);
        return s;
    };
    if (hipSetDevice(opts->device) != hipSuccess) return bail(CLLM_ERR_DEVICE);
    cllm_status s;
    if ((s = scratch_setup(c, opts->device))) return bail(s);
    const size_t E = c->elem;
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
    const size_t kv = c->kv_seq * c->max_batch * E;
    if ((s = dalloc(c, &c->kc, kv))) return bail(s);
    if ((s = dalloc(c, &c->vt, kv))) return bail(s);
    const int h2 = c->hd / 2;
    if ((s = dalloc_t(c, &c->rcos, (size_t)c->ctx_alloc * h2))) return bail(s);
    if ((s = dalloc_t(c, &c->rsin, (size_t)c->ctx_alloc * h2))) return bail(s);
    if (opts->workspace) {
        // the caller's device buffer: device memory of this context's GPU
        hipPointerAttribute_t a{};
        if (hipPointerGetAttributes(&a, opts->workspace) != hipSuccess || a.type != hipMemoryTypeDevice ||
            a.device != opts->device) {
            (void)hipGetLastError();
            return bail(CLLM_ERR_ARG);
        }
        c->ws_base = static_cast<uint8_t *>(opts->workspace);
        c->ws_size = opts->workspace_bytes;
        if (reinterpret_cast<uintptr_t>(c->ws_base) % kWsAlign != 0) return bail(CLLM_ERR_ARG);
    }
    if ((s = place_workspace(c))) return bail(s);

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
    return load_weights(c, WeightSource{tensors, 0});
}

cllm_status cllm_model_init_random(const cllm_config *cfg, uint64_t seed, const cllm_runtime_opts *opts,
                                   cllm_ctx **out) {
    if (!out) return CLLM_ERR_ARG;
    cllm_status s = cllm_model_create(cfg, opts, out);
    if (s) return s;
    if ((s = load_weights(*out, WeightSource{nullptr, seed}))) {
        cllm_model_free(*out);
        *out = nullptr;
    }
    return s;
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
    cllm_status s;
    if ((s = check_ctx(c)) || (s = check_seq(c, seq))) return s;
    if (!prompt || !first_token || len < 1) return fail(c, CLLM_ERR_ARG, "bad prompt");
    if (len + 1 > c->opts.max_ctx) return fail(c, CLLM_ERR_CAPACITY, "prompt of %d exceeds max_ctx", len);
    if ((s = check_ids(c, prompt, len))) return s;
    if ((s = prefill_impl(c, seq, prompt, len))) return s;
    std::vector<Ctl> h(c->max_batch);
    if ((s = read_ctl(c, h.data()))) return s;
    if (h[seq].err) return numeric_fail(c, seq, " in the prefill");
    if (c->dbg_on && c->dbg_host) {  // rows of the last chunk's last 64-row tile, to host rows 0..
        const int last = (len - 1) % c->pchunk;
        const int r0 = last / kMaxRows * kMaxRows;
        HIPCHK(c, hipMemcpy(c->dbg_host, c->dbg + (size_t)r0 * c->V, (size_t)(last + 1 - r0) * c->V * 4,
                            hipMemcpyDeviceToHost));
    }
    c->slot[seq].prefilled = true;
    c->slot[seq].L = h[seq].L;
    c->slot[seq].pending = h[seq].pending;
    *first_token = h[seq].pending;
    return CLLM_OK;
}

cllm_status cllm_jacobi_step(cllm_ctx *c, int32_t seq, const int32_t *block_in, int32_t m, int32_t *block_out,
                             int32_t *accepted_len) {
    if (!c) return CLLM_ERR_ARG;
    cllm_status s;
    if ((s = check_ctx(c)) || (s = check_seq(c, seq))) return s;
    return step_batch_impl(c, 1, &seq, block_in, m, &m, block_out, m, accepted_len);
}

cllm_status cllm_jacobi_step_batch(cllm_ctx *c, int32_t B, const int32_t *seq_ids, const int32_t *blocks_in,
                                   const int32_t *m, int32_t *blocks_out, int32_t *accepted) {
    if (!c) return CLLM_ERR_ARG;
    cllm_status s;
    if ((s = check_ctx(c))) return s;
    return step_batch_impl(c, B, seq_ids, blocks_in, c->opts.max_block, m, blocks_out, c->opts.max_block, accepted);
}

cllm_status cllm_jacobi_decode(cllm_ctx *c, int32_t seq, const int32_t *prompt, int32_t len, int32_t n,
                               int32_t max_new, const cllm_guess_spec *guess, int32_t *out_tokens,
                               cllm_decode_stats *stats) {
    if (!c) return CLLM_ERR_ARG;
    cllm_status s;
    if ((s = check_ctx(c)) || (s = check_seq(c, seq))) return s;
    if (!prompt || !out_tokens || len < 1) return fail(c, CLLM_ERR_ARG, "bad prompt or output");
    return decode_batch_impl(c, 1, &seq, prompt, &len, n, max_new, guess, out_tokens, stats);
}

cllm_status cllm_ar_decode(cllm_ctx *c, int32_t seq, const int32_t *prompt, int32_t len, int32_t max_new,
                           int32_t *out_tokens, cllm_decode_stats *stats) {
    if (!c) return CLLM_ERR_ARG;
    cllm_status s;
    if ((s = check_ctx(c)) || (s = check_seq(c, seq))) return s;
    if (!prompt || !out_tokens || len < 1) return fail(c, CLLM_ERR_ARG, "bad prompt or output");
    cllm_guess_spec g{};
    return decode_batch_impl(c, 1, &seq, prompt, &len, 1, max_new, &g, out_tokens, stats);
}

cllm_status cllm_jacobi_decode_batch(cllm_ctx *c, int32_t B, const int32_t *seq_ids, const int32_t *prompts,
                                     const int32_t *lens, int32_t n, int32_t max_new, const cllm_guess_spec *guesses,
                                     int32_t *out_tokens, cllm_decode_stats *stats) {
    if (!c) return CLLM_ERR_ARG;
    cllm_status s;
    if ((s = check_ctx(c))) return s;
    return decode_batch_impl(c, B, seq_ids, prompts, lens, n, max_new, guesses, out_tokens, stats);
}

cllm_status cllm_reset(cllm_ctx *c, int32_t seq) {
    if (!c) return CLLM_ERR_ARG;
    cllm_status s;
    if ((s = check_seq(c, seq))) return s;
    c->slot[seq] = cllm_ctx::Slot{};
    return CLLM_OK;
}

cllm_status cllm_debug_logits(cllm_ctx *c, int32_t enable, float *host_buf, size_t host_floats) {
    if (!c) return CLLM_ERR_ARG;
    if (enable) {
        if (!host_buf || host_floats < (size_t)c->dbg_rows * c->V)
            return fail(c, CLLM_ERR_ARG, "debug buffer needs %zu floats", (size_t)c->dbg_rows * c->V);
        if (!c->dbg) {  // device logits of up to the row capacity (a prefill chunk's rows too), on first use
            cllm_status s = check_ctx(c);
            if (s || (s = dalloc_t(c, &c->dbg, (size_t)c->cap * c->V))) return s;
        }
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

cllm_status cllm_trace_enable(cllm_ctx *c, int32_t enable) {
    if (!c) return CLLM_ERR_ARG;
    cllm_status s;
    if ((s = check_ctx(c))) return s;
    if (enable && !c->trace_dev) {
        const size_t n = (size_t)c->max_batch * c->opts.max_new * kTraceStride;
        if ((s = dalloc_t(c, &c->trace_dev, n))) return s;
    }
    c->trace_on = enable != 0;
    return CLLM_OK;
}

cllm_status cllm_trace_read(cllm_ctx *c, int32_t seq, int32_t *records, int64_t cap, int64_t *n_records) {
    if (!c || !n_records || cap < 0 || (cap > 0 && !records)) return CLLM_ERR_ARG;
    cllm_status s;
    if ((s = check_seq(c, seq))) return s;
    const int64_t n = std::min<int64_t>(cap, c->slot[seq].trace_n);
    *n_records = c->slot[seq].trace_n;
    if (n > 0)
        HIPCHK(c, hipMemcpy(records, c->trace_dev + (size_t)seq * c->opts.max_new * kTraceStride,
                            (size_t)n * kTraceStride * sizeof(int32_t), hipMemcpyDeviceToHost));
    return CLLM_OK;
}

cllm_status cllm_trace_count(const int32_t *records, int64_t n_records, const int32_t *tokens, int64_t n_tokens,
                             int32_t n, int32_t block_policy, cllm_trace_stats *out) {
    if (!out || n_records < 0 || n_tokens < 0 || (n_records > 0 && (!records || !tokens)) || n < 1 ||
        n > kMaxBlock || (block_policy != 0 && block_policy != 1))
        return CLLM_ERR_ARG;
    memset(out, 0, sizeof(*out));
    auto rec = [&](int64_t t) { return records + t * kTraceStride; };
    // acceptance iteration of every output position, and the records' sanity
    std::vector<int64_t> acc((size_t)n_tokens, -1);
    int64_t a_sum = 0;
    std::vector<int32_t> starts;
    for (int64_t t = 0; t < n_records; ++t) {
        const int32_t *r = rec(t);
        const int32_t e = r[1], m = r[3], a = r[4];
        if (m < 1 || m > n || a < 1 || a > m || e < 0 || (int64_t)e + a > n_tokens) return CLLM_ERR_ARG;
        for (int32_t q = e; q < e + a; ++q) acc[q] = t;
        a_sum += a;
        if (starts.empty() || starts.back() != r[2]) starts.push_back(r[2]);
    }
    // stationary: walking back from the iteration before q's acceptance while q's prediction
    // is its final token, some iteration has q past its next pending position
    int64_t stationary = 0;
    for (int64_t q = 0; q < n_tokens; ++q) {
        for (int64_t t = acc[q] - 1; t >= 0; --t) {
            const int32_t *r = rec(t);
            const int64_t k = q - r[1] - 1;
            if (k < 0 || k >= r[3] || r[5 + kMaxBlock + k] != tokens[q]) break;
            if (q >= (int64_t)r[1] + r[4] + 1) {
                ++stationary;
                break;
            }
        }
    }
    out->iterations = n_records;
    out->fast_forward_mean = n_records ? (double)a_sum / (double)n_records : 0.0;
    out->stationary = stationary;
    out->windows = block_policy == 0 ? (int64_t)starts.size() : (n_tokens + n - 1) / n;
    out->stationary_per_window = out->windows ? (double)stationary / (double)out->windows : 0.0;
    return CLLM_OK;
}

cllm_status cllm_collect_states(const int32_t *records, int64_t n_records, const int32_t *tokens, int64_t n_tokens,
                                int32_t n, double rate, uint64_t seed, int32_t *states, int32_t *augmented,
                                int32_t *block_start, int64_t cap, int64_t *n_states) {
    if (!n_states || n_records < 0 || n_tokens < 0 || cap < 0 || (n_records > 0 && (!records || !tokens)) ||
        (cap > 0 && (!states || !augmented || !block_start)) || n < 1 || n > kMaxBlock || !(rate >= 0.0 && rate <= 1.0))
        return CLLM_ERR_ARG;
    const uint64_t thr = (uint64_t)std::nearbyint(rate * 9007199254740992.0);  // rate * 2^53, ties to even
    int64_t count = 0;
    std::vector<int32_t> st((size_t)n), fx((size_t)n);
    auto emit = [&](int32_t b0, int32_t nb) {
        if (count < cap) {
            int32_t *so = states + count * n, *ao = augmented + count * n;
            for (int32_t i = 0; i < n; ++i) so[i] = ao[i] = i < nb ? st[i] : -1;
            for (int32_t i = 0; i < nb; ++i)
                if (ao[i] != fx[i] && (splitmix64(splitmix64(splitmix64(seed) ^ (uint64_t)count) ^ (uint64_t)i) >> 11) < thr)
                    ao[i] = fx[i];
            block_start[count] = b0;
        }
        ++count;
    };
    int64_t t = 0;
    while (t < n_records) {
        const int32_t *r0 = records + t * kTraceStride;
        const int32_t b0 = r0[2], nb = r0[3];
        if (r0[1] != b0 || nb < 1 || nb > n || (int64_t)b0 + nb > n_tokens) return CLLM_ERR_ARG;
        for (int32_t i = 0; i < nb; ++i) fx[i] = tokens[b0 + i];
        for (; t < n_records && records[t * kTraceStride + 2] == b0; ++t) {
            const int32_t *rc = records + t * kTraceStride;
            const int32_t e = rc[1], m = rc[3];
            if (e < b0 || e - b0 + m != nb) return CLLM_ERR_ARG;  // the block's state is fixed tokens + z
            for (int32_t i = 0; i < e - b0; ++i) st[i] = tokens[b0 + i];
            for (int32_t k = 0; k < m; ++k) st[e - b0 + k] = rc[5 + k];
            emit(b0, nb);
        }
        for (int32_t i = 0; i < nb; ++i) st[i] = fx[i];
        emit(b0, nb);  // the fixed point closes the trajectory
    }
    *n_states = count;
    return CLLM_OK;
}

cllm_status cllm_loss_head(cllm_ctx *c, const float *teacher, const float *student, int32_t n_pairs,
                           const float *ar_rows, const int32_t *ar_targets, int32_t n_ar, float omega, float *row_kl,
                           float *row_nll, float *d_student, float *d_ar, float *d_weight, double *loss) {
    if (!c || !loss || !loss_args_ok(teacher, student, n_pairs, ar_rows, ar_targets, n_ar, omega, row_kl, row_nll,
                                     d_student, d_ar))
        return c ? fail(c, CLLM_ERR_ARG, "loss head: bad arguments (pairs + AR rows in [1, 64])") : CLLM_ERR_ARG;
    cllm_status s;
    if ((s = check_ctx(c))) return s;
    if (!c->w_lm) return fail(c, CLLM_ERR_STATE, "loss head: weights not set");
    for (int i = 0; i < n_ar; ++i)
        if (ar_targets[i] < 0 || ar_targets[i] >= c->V) return fail(c, CLLM_ERR_ARG, "loss head: target out of range");
    const int P = n_pairs, A = n_ar, Rg = P + A, d = c->d, V = c->V;
    auto &w = c->loss;
    // staging of the host arrays: rows (teacher, student, AR), targets, per-row losses, dH, loss
    if ((s = loss_buf(c, &w.H, &w.h, (size_t)(2 * P + A) * d)) || (s = loss_buf(c, &w.out, &w.rows, (size_t)Rg)) ||
        (s = loss_buf(c, &w.dH, &w.dh, (size_t)Rg * d)) || (d_weight && (s = loss_buf(c, &w.dW, &w.dw, (size_t)V * d))))
        return s;
    if (!w.tg && (s = dalloc_t(c, &w.tg, (size_t)64))) return s;
    if (!w.loss && (s = dalloc_t(c, &w.loss, 1))) return s;
    hipStream_t st = c->stream;
    const size_t row_b = (size_t)d * sizeof(float);
    float *T = w.H, *S = w.H + (size_t)P * d, *Ar = w.H + (size_t)2 * P * d;
    if (P) {
        HIPCHK(c, hipMemcpyAsync(T, teacher, P * row_b, hipMemcpyHostToDevice, st));
        HIPCHK(c, hipMemcpyAsync(S, student, P * row_b, hipMemcpyHostToDevice, st));
    }
    if (A) {
        HIPCHK(c, hipMemcpyAsync(Ar, ar_rows, A * row_b, hipMemcpyHostToDevice, st));
        HIPCHK(c, hipMemcpyAsync(w.tg, ar_targets, A * sizeof(int32_t), hipMemcpyHostToDevice, st));
    }
    if ((s = loss_head_enqueue(c, T, S, P, Ar, w.tg, A, omega, w.out, w.out + P, w.dH, w.dH + (size_t)P * d,
                               d_weight ? w.dW : nullptr, w.loss)))
        return s;
    std::vector<float> rl((size_t)Rg);
    HIPCHK(c, hipMemcpyAsync(rl.data(), w.out, Rg * sizeof(float), hipMemcpyDeviceToHost, st));
    if (P) HIPCHK(c, hipMemcpyAsync(d_student, w.dH, P * row_b, hipMemcpyDeviceToHost, st));
    if (A) HIPCHK(c, hipMemcpyAsync(d_ar, w.dH + (size_t)P * d, A * row_b, hipMemcpyDeviceToHost, st));
    if (d_weight) HIPCHK(c, hipMemcpyAsync(d_weight, w.dW, (size_t)V * row_b, hipMemcpyDeviceToHost, st));
    HIPCHK(c, hipMemcpyAsync(loss, w.loss, sizeof(double), hipMemcpyDeviceToHost, st));
    HIPCHK(c, hipStreamSynchronize(st));
    for (int i = 0; i < P; ++i) row_kl[i] = rl[i];
    for (int i = 0; i < A; ++i) row_nll[i] = rl[P + i];
    return CLLM_OK;
}

cllm_status cllm_loss_head_device(cllm_ctx *c, const float *teacher, const float *student, int32_t n_pairs,
                                  const float *ar_rows, const int32_t *ar_targets, int32_t n_ar, float omega,
                                  float *row_kl, float *row_nll, float *d_student, float *d_ar, float *d_weight,
                                  double *loss) {
    if (!c || !loss_args_ok(teacher, student, n_pairs, ar_rows, ar_targets, n_ar, omega, row_kl, row_nll, d_student,
                            d_ar))
        return c ? fail(c, CLLM_ERR_ARG, "loss head: bad arguments (pairs + AR rows in [1, 64])") : CLLM_ERR_ARG;
    cllm_status s;
    if ((s = check_ctx(c))) return s;
    if (!c->w_lm) return fail(c, CLLM_ERR_STATE, "loss head: weights not set");
    const void *ptrs[] = {teacher, student, ar_rows, ar_targets, row_kl, row_nll, d_student, d_ar, d_weight, loss};
    for (const void *q : ptrs)
        if (q && !device_accessible(c, q))
            return fail(c, CLLM_ERR_ARG, "loss head (device): an array is not device memory of this context's GPU");
    return loss_head_enqueue(c, teacher, student, n_pairs, ar_rows, ar_targets, n_ar, omega, row_kl, row_nll,
                             d_student, d_ar, d_weight, loss);
}

cllm_status cllm_hidden_rows(cllm_ctx *c, int32_t seq, const int32_t *block, int32_t m, float *rows_out) {
    if (!c) return CLLM_ERR_ARG;
    cllm_status s;
    if ((s = check_ctx(c)) || (s = check_seq(c, seq))) return s;
    if (!block || !rows_out) return fail(c, CLLM_ERR_ARG, "NULL pointer");
    if (m < 1 || m > c->opts.max_block) return fail(c, CLLM_ERR_ARG, "m=%d outside [1, max_block]", m);
    if (!c->slot[seq].prefilled) return fail(c, CLLM_ERR_STATE, "hidden rows before prefill (slot %d)", seq);
    if ((s = check_ids(c, block, m))) return s;
    if (c->slot[seq].L + m > c->opts.max_ctx) return fail(c, CLLM_ERR_CAPACITY, "L + m exceeds max_ctx");
    auto &w = c->loss;
    if ((s = loss_buf(c, &w.hid, &w.hd_n, (size_t)m * c->d))) return s;
    // the decoder layers over the block at the committed length (provisional KV rows, no commit)
    if ((s = setup(c, MODE_STEP, 1, &seq, &m, block, m, 0))) return s;
    IterShape sh{m, 1, m, ceil_div(c->slot[seq].L + m, kAttnChunk), false, -1};
    sh.tail = false;
    if ((s = enqueue_iteration(c, sh, nullptr, nullptr))) return s;
    HIPCHK(c, launch_hidden_rows(c->X, c->d, m, c->d, c->g_final, c->cfg.rms_eps, w.hid, c->stream));
    HIPCHK(c, hipMemcpyAsync(rows_out, w.hid, (size_t)m * c->d * sizeof(float), hipMemcpyDeviceToHost, c->stream));
    HIPCHK(c, hipStreamSynchronize(c->stream));
    return CLLM_OK;
}

cllm_status cllm_hidden_rows_noalloc(cllm_ctx *c, int32_t seq, const int32_t *block, int32_t m, float *rows_out) {
    if (!c) return CLLM_ERR_ARG;
    cllm_status s;
    if ((s = check_ctx(c)) || (s = check_seq(c, seq))) return s;
    if (!block || !rows_out) return fail(c, CLLM_ERR_ARG, "NULL pointer");
    if (m < 1 || m > c->opts.max_block) return fail(c, CLLM_ERR_ARG, "m=%d outside [1, max_block]", m);
    if ((size_t)m * c->d > kNoAllocFloats)
        return fail(c, CLLM_ERR_CAPACITY, "hidden rows (no allocation): %d rows x %d floats exceed the %zu-float scratch",
                    m, c->d, kNoAllocFloats);
    if (!c->slot[seq].prefilled) return fail(c, CLLM_ERR_STATE, "hidden rows before prefill (slot %d)", seq);
    if ((s = check_ids(c, block, m))) return s;
    if (c->slot[seq].L + m > c->opts.max_ctx) return fail(c, CLLM_ERR_CAPACITY, "L + m exceeds max_ctx");
    float *hid = scratch_of(c->opts.device);
    if (!hid) return fail(c, CLLM_ERR_STATE, "no scratch address for device %d", c->opts.device);
    // as cllm_hidden_rows, with the staging rows in the device's scratch
    if ((s = setup(c, MODE_STEP, 1, &seq, &m, block, m, 0))) return s;
    IterShape sh{m, 1, m, ceil_div(c->slot[seq].L + m, kAttnChunk), false, -1};
    sh.tail = false;
    if ((s = enqueue_iteration(c, sh, nullptr, nullptr))) return s;
    HIPCHK(c, launch_hidden_rows(c->X, c->d, m, c->d, c->g_final, c->cfg.rms_eps, hid, c->stream));
    HIPCHK(c, hipMemcpyAsync(rows_out, hid, (size_t)m * c->d * sizeof(float), hipMemcpyDeviceToHost, c->stream));
    HIPCHK(c, hipStreamSynchronize(c->stream));
    return CLLM_OK;
}

cllm_status cllm_seq_state(const cllm_ctx *c, int32_t seq, int32_t *committed_len, int32_t *pending) {
    if (!c || seq < 0 || seq >= c->max_batch || !committed_len || !pending) return CLLM_ERR_ARG;
    if (!c->slot[seq].prefilled) return CLLM_ERR_STATE;
    *committed_len = c->slot[seq].L;
    *pending = c->slot[seq].pending;
    return CLLM_OK;
}

cllm_status cllm_timing_enable(cllm_ctx *c, int32_t kernel_class, int32_t max_rows, int32_t every) {
    if (!c) return CLLM_ERR_ARG;
    if (kernel_class > CLLM_KT_LOSS_DW || max_rows < 0 || max_rows > kMaxRows || every < 1)
        return fail(c, CLLM_ERR_ARG, "unknown kernel class, bad max_rows or bad sampling stride");
    c->kt_class = kernel_class < 0 ? -1 : kernel_class;
    c->kt_rg = max_rows == 0 ? 0 : rows_to_rg(max_rows);
    c->kt_every = every;
    c->kt_eligible = 0;
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
