// The weight-streaming GEMM of libcllm.so: its tile counts, parameter block and launcher.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cllm {

struct RowTab;
struct RowInfo;

constexpr int kLmTiles = 4;   // 16-column tiles per workgroup: LM head
constexpr int kNtQkv = 3;     // QKV (each tile holds rotate-half partners; 256 workgroups at 7B)
constexpr int kNtGateUp = 6;  // gate/up ((gate, up) tile pairs; 229 workgroups at 7B, one per CU)
constexpr int kNtResid = 1;   // O projection
constexpr int kDownSplits = 4;  // down projection: K split over 4 workgroups per 64-column group
constexpr int kGemmDepth = 2; // k-steps in flight per wave
constexpr int kPromptRows = 128;  // prompt GEMM: its largest row tile (the row capacity is a multiple)

enum GemmKind { GEMM_QKV = 0, GEMM_O = 1, GEMM_GATE_UP = 2, GEMM_DOWN = 3, GEMM_LM = 4, GEMM_LOGITS = 5 };

// Rows of an iteration: the row table, its per-row entries and the row capacity of the
// activation buffers (their plane size).
struct RowsRef {
    const RowTab *tab;
    const RowInfo *rows;
    int cap;
};

struct GemmParams {
    const uint8_t *W;  // packed tiles
    int Ks;            // k-steps per 16-row tile
    int cols;          // packed output columns (multiple of 16; of 32 for gate/up)
    int n_wg;          // workgroups along the columns (set by the launcher: ceil(cols / (16 NT)))
    int rt0;           // first row tile
    int row_tiles;     // row tiles of the launch (set by the launcher)
    const void *A;     // activation operand, packed operand order, lda elements per row
    int lda;
    RowsRef rr;
    // RMSNorm row factor (QKV, gate/up, LM head): per-16-column sums of squares [row][T]
    const float *ssq;
    int T, K;
    float eps;
    // E_QKV: Q operand; K cache [seq][layer][pos][d] and transposed V cache [seq][layer][d][pos]
    // given for this layer of sequence slot 0, kv_seq elements apart per slot
    void *Q, *Kc, *Vt;
    size_t kv_seq;
    int ctx_alloc;
    const float *rcos, *rsin;
    int d, hd;
    // E_RESID (O) and the down product: X += Y (rows of ldx floats); next RMSNorm operand
    // An = X (.) gain; its per-16-column sums of squares. The down product's Y is summed from
    // kDownSplits K-split partial products in `part` (kDownSplits x row capacity x ldx floats).
    float *Xout, *ssq_out;
    int ldx;
    const float *gain;
    void *An;
    float *part;
    // class-pair K split of multi-row products (bf16): four planes of t_c = x_c + x_(c+4), each
    // row capacity x cols floats, in the MFMA's C layout per 16 x 16 block
    float *spart;
    // the RMSNorm row factors of those products' rows [row capacity], written by the split launch
    float *sinv;
    // E_SWIGLU
    void *H;
    int Fp;
    // E_ARGMAX: per-workgroup (max, index) [workgroup][row capacity]; optional logits [row][V]
    float *pmax;
    int *pidx;
    float *dbg;
    int V;
    // E_LOGITS (plain fp32 products, no RMSNorm row factor): Zout[row][ldz], columns < V. With
    // kc > 0 the launch splits K: grid z takes k-steps [z kc, min((z + 1) kc, Ks)) and writes its
    // partial products to Zout + z * zstride.
    float *Zout;
    int ldz;
    int kc;
    size_t zstride;
    // launches of several row tiles (bf16): 0 = the row-tiled kernel; 1 = gemm_kernel over the
    // row tiles (the same values; kept as the reference of the kernel driver's check)
    int tile_kernel;
};

// Launch a product of `kind` over row_tiles tiles of 16 * rg rows (rg = 4 when row_tiles > 1);
// e0 / e1 (optional) time the launch.
hipError_t launch_gemm(GemmKind kind, bool bf16, int rg, int row_tiles, const GemmParams &p, hipStream_t s,
                       hipEvent_t e0, hipEvent_t e1);

// Prompt (prefill) product of `kind` (QKV, O, gate/up, down) over `rows` rows (bf16 models):
// workgroup tiles of up to kPromptRows rows with operands shared through LDS; every prompt row
// takes this path, so its values do not depend on the chunking. O and down run as fixed K ranges
// (2 and 4) into fp32 partials, then a reduction with the residual epilogue. The row capacity
// must be a multiple of kPromptRows.
hipError_t launch_gemm_prompt(GemmKind kind, int rows, const GemmParams &p, hipStream_t s, hipEvent_t e0,
                              hipEvent_t e1);

}  // namespace cllm
