// Kernel parameter blocks and launchers of libcllm.so (host and device).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cllm {

struct Ctl;

constexpr int kLmTiles = 4;  // 16-column tiles per LM-head workgroup

enum GemmKind { GEMM_QKV = 0, GEMM_O = 1, GEMM_GATE_UP = 2, GEMM_DOWN = 3, GEMM_LM = 4 };

struct GemmParams {
    const uint8_t *W;  // packed tiles
    int Ks;            // k-steps per 16-row tile
    int n_wg;          // workgroups (tiles / NT)
    // activation operand
    const void *A;     // compute dtype, rows of lda elements (A_ACT)
    int lda;
    const float *X;    // fp32 residual stream, rows of ldx floats (A_NORM reads it; E_RESID updates it)
    int ldx;
    const float *gain; // RMSNorm gain [K]
    const float *ssq;  // per-16-column sums of squares [T][kMaxRows]
    int T, K;
    float eps;
    const Ctl *ctl;
    // E_QKV
    void *Q, *Kc, *Vt;
    int ctx_alloc;
    const float *rcos, *rsin;
    int d, hd;
    // E_RESID
    float *Xout, *ssq_out;
    // E_SWIGLU
    void *H;
    int Fp;
    // E_ARGMAX
    float *pmax;
    int *pidx;
    float *dbg;
    int V;
};

struct EmbedParams {
    const void *E;
    float *X, *ssq;
    int d;
    const Ctl *ctl;
};

struct AttnParams {
    const void *Q, *Kc, *Vt;
    void *O;
    float *Opart, *Mpart, *Lpart;
    int d, hd, n_heads, nch, ctx_alloc;
    float scale_log2;
    const Ctl *ctl;
};

struct ScanParams {
    Ctl *ctl;
    const float *pmax;
    const int *pidx;
    int n_wg;
    int32_t *out;           // decode output tokens
    const int32_t *stream;  // guess stream (may be null)
    int advance_only;       // prefill chunk without LM head: commit all rows, no predictions
};

// Host-side edits of the control block, applied on the stream in order with the kernels.
struct SetupParams {
    Ctl *ctl;
    int mode, m, set_L, L;
    int32_t z[64];
};
hipError_t launch_setup(const SetupParams &p, hipStream_t s);

hipError_t launch_gemm(GemmKind kind, bool bf16, int rg, int nt_qkv, const GemmParams &p, hipStream_t s,
                       hipEvent_t e0, hipEvent_t e1);
hipError_t launch_embed(bool bf16, int rows, const EmbedParams &p, hipStream_t s, hipEvent_t e0, hipEvent_t e1);
hipError_t launch_attn(bool bf16, int rg, int nch_launch, const AttnParams &p, hipStream_t s, hipEvent_t e0,
                       hipEvent_t e1);
hipError_t launch_attn_combine(bool bf16, int rows, const AttnParams &p, hipStream_t s, hipEvent_t e0,
                               hipEvent_t e1);
hipError_t launch_scan(const ScanParams &p, hipStream_t s, hipEvent_t e0, hipEvent_t e1);
hipError_t launch_decode_init(const ScanParams &p, hipStream_t s);
hipError_t launch_repack(bool bf16, const void *src, const int32_t *perm, int K, int Ks, int n_tiles, uint8_t *dst,
                         hipStream_t s);

}  // namespace cllm
