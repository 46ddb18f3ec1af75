// Kernel parameter blocks and launchers of libcllm.so (host and device).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cllm {

struct Ctl;

constexpr int kLmTiles = 4;   // 16-column tiles per workgroup: LM head
constexpr int kNtQkv = 4;     // QKV (pairs of rotate-half partner tiles)
constexpr int kNtGateUp = 2;  // gate/up ((gate, up) tile pairs)
constexpr int kNtResid = 1;   // O and down projections
constexpr int kGemmDepth = 2; // k-steps in flight per wave
constexpr bool kGemmKContig = false;  // k-steps per wave: interleaved (false) or contiguous

enum GemmKind { GEMM_QKV = 0, GEMM_O = 1, GEMM_GATE_UP = 2, GEMM_DOWN = 3, GEMM_LM = 4 };

struct GemmParams {
    const uint8_t *W;  // packed tiles
    int Ks;            // k-steps per 16-row tile
    int n_wg;          // workgroups (tiles / NT)
    const void *A;     // activation operand (compute dtype), rows of lda elements
    int lda;
    // RMSNorm row factor (QKV, gate/up, LM head): per-16-column sums of squares [row][T]
    const float *ssq;
    int T, K;
    float eps;
    const Ctl *ctl;
    // E_QKV
    void *Q, *Kc, *Vt;
    int ctx_alloc;
    const float *rcos, *rsin;
    int d, hd;
    // E_RESID: X += Y (rows of ldx floats); next RMSNorm operand An = X (.) gain; new partials
    float *Xout, *ssq_out;
    int ldx;
    const float *gain;
    void *An;
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
    void *An;           // first RMSNorm operand X (.) gain
    const float *gain;
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

hipError_t launch_gemm(GemmKind kind, bool bf16, int rg, const GemmParams &p, hipStream_t s, hipEvent_t e0,
                       hipEvent_t e1);
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
