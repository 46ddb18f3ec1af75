// Kernel parameter blocks and launchers of libcllm.so (host and device).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "gemm.h"

namespace cllm {

struct Ctl;
struct RowTab;
struct RowInfo;

struct EmbedParams {
    const void *E;
    float *X, *ssq;
    void *An;           // first RMSNorm operand X (.) gain
    const float *gain;
    int d;
    RowsRef rr;
};

struct AttnParams {
    const void *Q, *Kc, *Vt;  // caches as in GemmParams
    size_t kv_seq;
    void *O;
    float *Opart, *Mpart, *Lpart;  // [head][chunk][row capacity] (x hd for Opart)
    int d, hd, n_heads, nch, ctx_alloc;
    int nrb;  // workgroups per batch entry along its block rows (16 * rg rows each)
    float scale_log2;
    RowsRef rr;
};

struct ScanParams {
    Ctl *ctl;               // control blocks, one per sequence slot
    RowTab *tab;
    RowInfo *rows;
    int cap;                // row capacity
    const float *pmax;
    const int *pidx;
    int n_wg;
    int32_t *out;           // decode output tokens, out_stride per slot
    const int32_t *stream;  // guess streams (may be null), stream_stride per slot
    int out_stride, stream_stride;
    int advance_only;       // prefill chunk without LM head: commit all rows, no predictions
    uint64_t advance_mask;  // prefill: bit b set = entry b's chunk does not end its prompt (commit only)
    int plan_inline;        // one batch entry: the scan also lays out the next row table
    int32_t *mlog;          // block size of each decode iteration (out_stride entries per slot), or null
    int32_t *trace;         // decode trajectory records (trace_cap per slot, kTraceStride int32 each), or null
    int trace_cap;
};

// Host-side edits of the control blocks and the row table, applied on the stream in order with
// the kernels. Entry b's tokens are zin[b * zstride + i], or with packed set zin[r0_b + i] (r0_b:
// the rows of the entries before it); a prefill pass may hold up to the row capacity.
struct SetupParams {
    Ctl *ctl;
    RowTab *tab;
    RowInfo *rows;
    const int32_t *zin;
    int zstride, nseq, mode, packed;
    uint64_t reset_mask;  // bit b: entry b starts a prompt (L = 0, error and done flags cleared)
    int32_t seq[64], m[64];
};

// Lay out the row table from the control blocks of the batch entries already in the table.
struct PlanParams {
    Ctl *ctl;
    RowTab *tab;
    RowInfo *rows;
    int cap;
};

hipError_t launch_setup(const SetupParams &p, hipStream_t s);

hipError_t launch_embed(bool bf16, int rows, const EmbedParams &p, hipStream_t s, hipEvent_t e0, hipEvent_t e1);
hipError_t launch_attn(bool bf16, int rg, int nch_launch, int nseq_launch, const AttnParams &p, hipStream_t s,
                       hipEvent_t e0, hipEvent_t e1);
hipError_t launch_attn_combine(bool bf16, int rows, const AttnParams &p, hipStream_t s, hipEvent_t e0,
                               hipEvent_t e1);
// One-kernel attention: nrg 16-row groups per batch entry, no row seeing more than
// kFusedChunks 64-key chunks, head_dim <= 128 (O written directly; bit-identical to
// launch_attn + combine).
constexpr int kFusedChunks = 32;
hipError_t launch_attn_fused(bool bf16, int nrg, int nseq_launch, const AttnParams &p, hipStream_t s, hipEvent_t e0,
                             hipEvent_t e1);
hipError_t launch_scan(int nseq_launch, const ScanParams &p, hipStream_t s, hipEvent_t e0, hipEvent_t e1);
hipError_t launch_decode_init(int nseq, const ScanParams &p, hipStream_t s);
hipError_t launch_plan(const PlanParams &p, hipStream_t s);
// CLLM loss head (global consistency KL + omega AR loss at the LM head) and its gradients.
struct LossParams {
    const float *Z;    // logits [R][ldz]: teacher rows 0..P-1, student rows P..2P-1, AR rows 2P..
    const int32_t *targets;  // AR targets [A]
    int P, A, V, ldz;
    float omega;
    float *kl, *nll;   // per pair / per AR row
    float *D;          // logit gradients [P + A][ldz] (student rows, then AR rows; 0 past V)
};
// Per-row losses and logit gradients in two passes over vocabulary chunks of kLossChunk entries:
// per-chunk statistics (stats: [P + A][chunks][5] floats), then their combination in chunk order,
// the losses and D. e0 (if any) marks the start of the first pass.
constexpr int kLossChunk = 2048;
hipError_t launch_loss_rows(const LossParams &p, float *stats, hipStream_t s, hipEvent_t e0, hipEvent_t e1);
// Rows (fp32 [.][d]: np teacher rows T0, np student rows S0, na AR rows R0, in that order) to the
// two bf16 planes (or one fp32 plane) of a GEMM operand of row capacity cap; e0 marks its start.
hipError_t launch_pack_rows(bool bf16, const float *T0, const float *S0, int np, const float *R0, int na, int d,
                            int cap, void *A, hipStream_t s, hipEvent_t e0);
// D [rows][ldd] as the GEMM operand of dH = D W (Dact: operand order, row capacity cap, K = Vp);
// in bf16 also D^T and the gradient rows H (S0 rows < np, then R0) as the operands of dW = D^T H
// with the contraction over rpad rows (DT: 2 planes Vp x rpad; HT: 2 planes d x rpad; zero rows
// from `rows`). e1 marks the end of the last launch.
hipError_t launch_loss_pack(bool bf16, const float *D, int rows, int ldd, int Vp, int cap, void *Dact, int rpad,
                            uint16_t *DT, const float *S0, int np, const float *R0, int d, uint16_t *HT,
                            hipStream_t s, hipEvent_t e1);
// The packed LM head [Vp][d] repacked as the weight operand of dH = D W (tiles over k-steps of the
// vocabulary and 16 columns of d); Vp x d elements.
hipError_t launch_transpose_lm(bool bf16, const uint8_t *W, int Vp, int d, uint8_t *WT, hipStream_t s);
// dH from the K-split partials [nsplit][rows][d], summed in split order: rows < np to dS [np][d],
// the others to dA. e1 marks the end.
hipError_t launch_loss_dh_sum(const float *part, int nsplit, int rows, int d, int np, float *dS, float *dA,
                              hipStream_t s, hipEvent_t e1);
// dW[v][k] = sum_r D[r][v] H[r][k] for v < V (rows <= 64), H row r = S0 row r for r < np, else
// R0 row r - np: bf16 from the DT / HT operands, fp32 from D, S0 and R0.
hipError_t launch_loss_dw(bool bf16, const uint16_t *DT, const uint16_t *HT, int Vp, int rpad, const float *D,
                          int rows, int ldd, const float *S0, int np, const float *R0, int d, int V, float *dW,
                          hipStream_t s, hipEvent_t e0, hipEvent_t e1);
// LM-head input rows out[r] = x_r (.) g / sqrt(mean(x_r^2) + eps) of the residual rows X [rows][ldx]
// (the mean in a fixed order).
hipError_t launch_hidden_rows(const float *X, int ldx, int rows, int d, const float *g, float eps, float *out,
                              hipStream_t s);
// *loss = sum kl[0..np) + omega * sum nll[0..na), each in row order, in double (one thread).
hipError_t launch_loss_total(const float *kl, int np, const float *nll, int na, float omega, double *loss,
                             hipStream_t s);

// Seeded synthetic weights, drawn in place: kind 2 fills n floats with 1.0 (norm gains); kinds
// 0 (float) and 1 (bf16) fill n elements with std x a standard normal deviate: for element i,
// the Box-Muller pair j = i / 2 of the counter-based draws mix(key ^ 2j), mix(key ^ (2j + 1))
// (mix: SplitMix64's output function; u1 = (top 53 bits + 1) 2^-53, u2 = top 53 bits x 2^-53;
// r = sqrt(-2 ln u1); even i takes r cos(2 pi u2), odd i r sin(2 pi u2)), in double, rounded to
// fp32 and then (kind 1) to bf16, nearest even.
constexpr double kWeightStd = 0.02;
hipError_t launch_fill_weights(int kind, uint64_t key, double stdv, size_t n, void *out, hipStream_t s);
hipError_t launch_repack(bool bf16, const void *src, const int32_t *perm, int K, int Ks, int n_tiles, uint8_t *dst,
                         hipStream_t s);

}  // namespace cllm
