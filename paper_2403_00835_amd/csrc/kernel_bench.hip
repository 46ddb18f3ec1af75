// kernel_bench: standalone driver of libcllm's weight-streaming GEMM kernels at the LLaMA-2-7B
// shape (d 4096, FFN 11008, vocab 32000, head_dim 128, bf16) for one iteration of `rows` rows
// (more than 64 rows: row tiles of 64, as in batched iterations). With more than 64 rows the
// prompt GEMM (prefill passes: QKV, O, gate/up, down) is timed as well at the same row count.
//
// Each product of an iteration (QKV, O, gate/up, down, LM head) is launched `iters` times through
// the library's own launchers, in the library's launch configuration, over rotating copies of its
// packed weights inside a 2 GiB buffer, so no launch finds its weights in the last-level cache.
// A plain device copy of a known byte count runs first: it scales the hardware byte counters
// (rocprofv3 --pmc FETCH_SIZE, WRITE_SIZE) to bytes. A streaming read of 1 GiB follows: the
// practical HBM read ceiling the GEMMs are compared with. Weights and activations hold arbitrary
// finite values: the timing and the traffic of these kernels do not depend on them.
//
// Usage: kernel_bench [rows (1..512, default 16)] [iters (default 20)]
//        kernel_bench check [rows (1..512, default 160)]
// The check mode fills weights, operands and the RMSNorm inputs with seeded random values and
// runs each decode product (QKV, O, gate/up, down, LM head) twice over the same inputs, launched
// for the row tiles the rows fill and for at least two row tiles as batched iterations are: as the
// library launches it (with several row tiles: QKV, gate/up and the LM head through the
// class-pair K split, also when the live rows fit one tile, the down ranges through the row-tiled
// kernel, which then takes gemm_kernel's body) and through gemm_kernel over the same row tiles; every
// output (Q operand, cached keys and values, residual rows, next RMSNorm operand and its sums of
// squares, SwiGLU rows, the LM head's
// per-workgroup argmax values and indices) must be bit-identical.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <string>
#include <vector>

#include "device.h"
#include "launch.h"

using namespace cllm;

#define CK(x)                                                                                    \
    do {                                                                                         \
        hipError_t e_ = (x);                                                                     \
        if (e_ != hipSuccess) {                                                                  \
            std::fprintf(stderr, "kernel_bench: %s failed: %s\n", #x, hipGetErrorString(e_));   \
            std::exit(1);                                                                        \
        }                                                                                        \
    } while (0)

__global__ __launch_bounds__(256) void copy_known(const u32x4 *__restrict__ src, u32x4 *__restrict__ dst,
                                                  size_t n16) {
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += (size_t)gridDim.x * blockDim.x)
        dst[i] = src[i];
}

// Streaming read of n16 16-byte vectors (non-temporal loads, as the GEMMs stream their weights):
// the practical HBM read ceiling. The xor of the data is stored only if it equals a value it
// practically never takes, so the loads cannot be dropped and nothing is written.
__global__ __launch_bounds__(256) void stream_read(const u32x4 *__restrict__ src, size_t n16, uint32_t *out) {
    uint32_t acc = 0;
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += (size_t)gridDim.x * blockDim.x) {
        const u32x4 v = __builtin_nontemporal_load(src + i);
        acc ^= v.x ^ v.y ^ v.z ^ v.w;
    }
    if (acc == 0x9E3779B9u) out[0] = acc;
}

// Seeded fill: bf16 values of magnitude below `scale` (no NaN or infinity), or positive fp32
// values in [lo, lo + span).
__global__ void fill_bf16(uint16_t *x, size_t n, uint64_t seed, float scale) {
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
        const uint64_t h = mix64(seed ^ (i * 0x9E3779B97F4A7C15ull));
        const float u = (float)(h >> 40) * 0x1.0p-24f * 2.0f - 1.0f;
        x[i] = f2bf(u * scale);
    }
}
__global__ void fill_f32(float *x, size_t n, uint64_t seed, float lo, float span) {
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
        const uint64_t h = mix64(seed ^ (i * 0x9E3779B97F4A7C15ull));
        x[i] = lo + (float)(h >> 40) * 0x1.0p-24f * span;
    }
}

namespace {

constexpr int kD = 4096, kF = 11008, kV = 32000, kHd = 128, kCtx = 1024, kL = 512;
constexpr int kFp = (kF + 31) / 32 * 32;
constexpr size_t kWBytes = (size_t)2 << 30;

template <typename T>
T *dev(size_t count, int byte) {
    T *p = nullptr;
    CK(hipMalloc(&p, count * sizeof(T)));
    CK(hipMemset(p, byte, count * sizeof(T)));
    return p;
}

struct Shape {
    const char *name;
    GemmKind kind;
    int nt;    // 16-column tiles per workgroup
    int cols;  // packed output columns
    int K;
};

}  // namespace

int check_main(int rows);

int main(int argc, char **argv) {
    if (argc > 1 && std::string(argv[1]) == "check") return check_main(argc > 2 ? std::atoi(argv[2]) : 160);
    const int rows = argc > 1 ? std::atoi(argv[1]) : 16;
    const int iters = argc > 2 ? std::atoi(argv[2]) : 20;
    if (rows < 1 || rows > 512 || iters < 1) {
        std::fprintf(stderr, "usage: kernel_bench [rows 1..512] [iters >= 1]\n");
        return 2;
    }
    const int rg = rows <= 16 ? 1 : rows <= 32 ? 2 : 4;
    const int row_tiles = rows > kMaxRows ? (rows + kMaxRows - 1) / kMaxRows : 1;
    // row capacity of the activation buffers: whole decode row tiles and prompt-GEMM row tiles
    const int cap = (row_tiles * kMaxRows + kPromptRows - 1) / kPromptRows * kPromptRows;

    uint8_t *W = dev<uint8_t>(kWBytes, 0x11);  // bf16 0x1111 in every weight
    // one sequence (slot 0) with a block of `rows` rows at positions kL ..
    RowTab th{};
    th.R = rows;
    th.nseq = 1;
    th.m[0] = rows;
    th.L[0] = kL;
    RowTab *tab = dev<RowTab>(1, 0);
    CK(hipMemcpy(tab, &th, sizeof(RowTab), hipMemcpyHostToDevice));
    static RowInfo rh[512];
    for (int i = 0; i < cap; ++i) rh[i] = RowInfo{0, kL + i, 0, i};
    RowInfo *rinfo = dev<RowInfo>(cap, 0);
    CK(hipMemcpy(rinfo, rh, sizeof(RowInfo) * cap, hipMemcpyHostToDevice));
    // activation operands: two bf16 planes of cap rows (act_plane elements each)
    void *A_d = dev<uint16_t>(2 * act_plane(cap, kD), 0);
    void *A_f = dev<uint16_t>(2 * act_plane(cap, kFp), 0);
    void *An = dev<uint16_t>(2 * act_plane(cap, kD), 0);
    void *Q = dev<uint16_t>(2 * act_plane(cap, kD), 0);
    void *H = dev<uint16_t>(2 * act_plane(cap, kFp), 0);
    void *Kc = dev<uint16_t>((size_t)kCtx * kD, 0);
    void *Vt = dev<uint16_t>((size_t)kD * kCtx, 0);
    float *ssq = dev<float>((size_t)(kD / 16) * cap, 0);
    float *ssq_out = dev<float>((size_t)(kD / 16) * cap, 0);
    float *X = dev<float>((size_t)cap * kD, 0);
    float *gain = dev<float>(kD, 0);
    float *rcos = dev<float>((size_t)kCtx * (kHd / 2), 0);
    float *rsin = dev<float>((size_t)kCtx * (kHd / 2), 0);
    const int n_wg_lm = (kV + 16 * kLmTiles - 1) / (16 * kLmTiles);
    float *pmax = dev<float>((size_t)n_wg_lm * cap, 0);
    int *pidx = dev<int>((size_t)n_wg_lm * cap, 0);

    {  // 256 MiB copy: read 268435456 bytes, write 268435456 bytes, inside the weight buffer
        const size_t bytes = (size_t)256 << 20;
        hipLaunchKernelGGL(copy_known, dim3(4096), dim3(256), 0, 0, reinterpret_cast<const u32x4 *>(W),
                           reinterpret_cast<u32x4 *>(W + ((size_t)1 << 30)), bytes / 16);
        CK(hipGetLastError());
        CK(hipDeviceSynchronize());
        std::printf("copy_known: %zu bytes read, %zu bytes written\n", bytes, bytes);
    }

    {  // streaming-read ceiling: 1 GiB per launch, 2048 workgroups (8 per CU), 10 launches
        const size_t bytes = (size_t)1 << 30;
        uint32_t *sink = dev<uint32_t>(1, 0);
        hipEvent_t s0, s1;
        CK(hipEventCreate(&s0));
        CK(hipEventCreate(&s1));
        hipLaunchKernelGGL(stream_read, dim3(2048), dim3(256), 0, 0, reinterpret_cast<const u32x4 *>(W), bytes / 16, sink);
        CK(hipGetLastError());
        CK(hipEventRecord(s0, 0));
        for (int i = 0; i < 10; ++i)
            hipLaunchKernelGGL(stream_read, dim3(2048), dim3(256), 0, 0,
                               reinterpret_cast<const u32x4 *>(W + (size_t)(i & 1) * bytes), bytes / 16, sink);
        CK(hipGetLastError());
        CK(hipEventRecord(s1, 0));
        CK(hipEventSynchronize(s1));
        float ms = 0.0f;
        CK(hipEventElapsedTime(&ms, s0, s1));
        std::printf("stream_read: %zu bytes per launch, %.2f us/launch, %.1f GB/s\n", bytes, ms * 1e3 / 10,
                    bytes / (ms * 1e-3 / 10) / 1e9);
    }

    const Shape shapes[] = {
        {"qkv", GEMM_QKV, kNtQkv, 3 * kD, kD},
        {"o", GEMM_O, kNtResid, kD, kD},
        {"gate_up", GEMM_GATE_UP, kNtGateUp, 2 * kFp, kD},
        {"down", GEMM_DOWN, kLmTiles, kD, kFp},
        {"lm_head", GEMM_LM, kLmTiles, n_wg_lm * 16 * kLmTiles, kD},
    };
    float *part = dev<float>((size_t)kDownSplits * cap * kD, 0);  // K-split partials of the down product
    float *spart = dev<float>((size_t)4 * cap * std::max(2 * kFp, kV), 0);       // class-pair split partials
    float *sinv = dev<float>((size_t)cap, 0);                      // and their row factors
    hipEvent_t e0, e1;
    CK(hipEventCreate(&e0));
    CK(hipEventCreate(&e1));
    auto params = [&](const Shape &s) {
        GemmParams p{};
        p.Ks = s.K / 32;
        p.cols = s.cols;
        p.n_wg = (s.cols / 16 + s.nt - 1) / s.nt;  // as the launcher sets it
        p.A = s.kind == GEMM_DOWN ? A_f : A_d;
        p.lda = s.K;
        p.ssq = ssq;
        p.T = kD / 16;
        p.K = kD;
        p.eps = 1e-6f;
        p.rr = RowsRef{tab, rinfo, cap};
        p.Q = Q;
        p.Kc = Kc;
        p.Vt = Vt;
        p.ctx_alloc = kCtx;
        p.rcos = rcos;
        p.rsin = rsin;
        p.d = kD;
        p.hd = kHd;
        p.Xout = X;
        p.ssq_out = ssq_out;
        p.ldx = kD;
        p.gain = gain;
        p.An = An;
        p.H = H;
        p.Fp = kFp;
        p.pmax = pmax;
        p.pidx = pidx;
        p.dbg = nullptr;
        p.V = kV;
        p.part = part;
        p.spart = spart;
        p.sinv = sinv;
        return p;
    };
    // more than 32 rows: the products as iterations launch them (class-pair split, row-tiled
    // kernel), then gemm_kernel over the same row tiles for comparison
    for (int pass = 0; pass < (rg == 4 ? 2 : 1); ++pass)
    for (const Shape &s : shapes) {
        GemmParams p = params(s);
        p.tile_kernel = pass;
        if (pass == 1 && s.kind == GEMM_LM) continue;
        const size_t per = (size_t)(s.cols / 16) * p.Ks * kTileBytes;  // packed weight bytes per launch
        const int copies = (int)(kWBytes / per);
        if (copies < 2 || s.cols % 32 != 0) {
            std::fprintf(stderr, "kernel_bench: shape %s does not fit the buffers\n", s.name);
            return 1;
        }
        for (int i = 0; i < 2; ++i) {  // warm-up
            p.W = W + (size_t)(i % copies) * per;
            CK(launch_gemm(s.kind, true, rg, row_tiles, p, 0, nullptr, nullptr));
        }
        CK(hipDeviceSynchronize());
        CK(hipEventRecord(e0, 0));
        for (int i = 0; i < iters; ++i) {
            p.W = W + (size_t)((i + 2) % copies) * per;
            CK(launch_gemm(s.kind, true, rg, row_tiles, p, 0, nullptr, nullptr));
        }
        CK(hipEventRecord(e1, 0));
        CK(hipEventSynchronize(e1));
        float ms = 0.0f;
        CK(hipEventElapsedTime(&ms, e0, e1));
        const double us = ms * 1e3 / iters;
        const double flops = 2.0 * rows * s.cols * s.K;  // algorithmic (the MFMA work is twice: hi, lo)
        std::printf("%s%-8s rows=%d row_tiles=%d weights=%zu bytes  %8.2f us/launch  %7.1f GB/s  %7.1f TFLOP/s\n",
                    pass ? "tile " : "", s.name, rows, row_tiles, per, us, per / us / 1e3, flops / us / 1e6);
    }
    if (rows > kMaxRows) {
        for (int k = 0; k < 4; ++k) {  // QKV, O, gate/up, down
            const Shape &s = shapes[k];
            GemmParams p = params(s);
            const size_t per = (size_t)(s.cols / 16) * p.Ks * kTileBytes;
            const int copies = (int)(kWBytes / per);
            for (int i = 0; i < 2; ++i) {
                p.W = W + (size_t)(i % copies) * per;
                CK(launch_gemm_prompt(s.kind, rows, p, 0, nullptr, nullptr));
            }
            CK(hipDeviceSynchronize());
            CK(hipEventRecord(e0, 0));
            for (int i = 0; i < iters; ++i) {
                p.W = W + (size_t)((i + 2) % copies) * per;
                CK(launch_gemm_prompt(s.kind, rows, p, 0, nullptr, nullptr));
            }
            CK(hipEventRecord(e1, 0));
            CK(hipEventSynchronize(e1));
            float ms = 0.0f;
            CK(hipEventElapsedTime(&ms, e0, e1));
            const double us = ms * 1e3 / iters;
            const double flops = 2.0 * rows * s.cols * s.K;
            std::printf("prompt %-8s rows=%d weights=%zu bytes  %8.2f us/launch  %7.1f TFLOP/s (MFMA work: twice)\n",
                        s.name, rows, per, us, flops / us / 1e6);
        }
    }
    CK(hipDeviceSynchronize());
    std::printf("done\n");
    return 0;
}

// ------------------------------------------------------------------------------------------
// check mode
// ------------------------------------------------------------------------------------------
namespace {

template <typename T>
std::vector<T> to_host(const T *d, size_t n) {
    std::vector<T> h(n);
    CK(hipMemcpy(h.data(), d, n * sizeof(T), hipMemcpyDeviceToHost));
    return h;
}

template <typename T>
size_t count_diff(const std::vector<T> &a, const std::vector<T> &b) {
    size_t n = 0;
    for (size_t i = 0; i < a.size(); ++i) n += std::memcmp(&a[i], &b[i], sizeof(T)) != 0;
    return n;
}

}  // namespace

int check_main(int rows) {
    if (rows < 1 || rows > 512) {
        std::fprintf(stderr, "kernel_bench check: rows must lie in 1..512\n");
        return 2;
    }
    // launched for the row tiles the rows fill and, as batched iterations launch them, for at
    // least two (their live rows may fit in one)
    const int row_tiles = std::max(2, (rows + kMaxRows - 1) / kMaxRows), cap = row_tiles * kMaxRows;
    const int launch_tiles[2] = {(rows + kMaxRows - 1) / kMaxRows, row_tiles};
    const size_t nW = (size_t)std::max(2 * kFp, kV) * kD;  // the largest packed product (LM head), elements
    uint16_t *W = dev<uint16_t>(nW, 0);
    RowTab th{};
    th.R = rows;
    th.nseq = 1;
    th.m[0] = rows;
    th.L[0] = kL;
    RowTab *tab = dev<RowTab>(1, 0);
    CK(hipMemcpy(tab, &th, sizeof(RowTab), hipMemcpyHostToDevice));
    static RowInfo rh[512];
    for (int i = 0; i < cap; ++i) rh[i] = RowInfo{0, kL + i, 0, i};
    RowInfo *rinfo = dev<RowInfo>(cap, 0);
    CK(hipMemcpy(rinfo, rh, sizeof(RowInfo) * cap, hipMemcpyHostToDevice));
    const size_t nAd = 2 * act_plane(cap, kD), nAf = 2 * act_plane(cap, kFp);
    uint16_t *A_d = dev<uint16_t>(nAd, 0), *A_f = dev<uint16_t>(nAf, 0);
    float *ssq = dev<float>((size_t)(kD / 16) * cap, 0), *gain = dev<float>(kD, 0);
    float *rcos = dev<float>((size_t)kCtx * (kHd / 2), 0), *rsin = dev<float>((size_t)kCtx * (kHd / 2), 0);
    float *X0 = dev<float>((size_t)cap * kD, 0);
    const dim3 fg(1024), fb(256);
    hipLaunchKernelGGL(fill_bf16, fg, fb, 0, 0, W, nW, 1ull, 0.05f);
    hipLaunchKernelGGL(fill_bf16, fg, fb, 0, 0, A_d, nAd, 2ull, 1.0f);
    hipLaunchKernelGGL(fill_bf16, fg, fb, 0, 0, A_f, nAf, 3ull, 1.0f);
    hipLaunchKernelGGL(fill_f32, fg, fb, 0, 0, ssq, (size_t)(kD / 16) * cap, 4ull, 1.0f, 15.0f);
    hipLaunchKernelGGL(fill_f32, fg, fb, 0, 0, gain, (size_t)kD, 5ull, 0.5f, 1.0f);
    hipLaunchKernelGGL(fill_f32, fg, fb, 0, 0, rcos, (size_t)kCtx * (kHd / 2), 6ull, -1.0f, 2.0f);
    hipLaunchKernelGGL(fill_f32, fg, fb, 0, 0, rsin, (size_t)kCtx * (kHd / 2), 7ull, -1.0f, 2.0f);
    hipLaunchKernelGGL(fill_f32, fg, fb, 0, 0, X0, (size_t)cap * kD, 8ull, -2.0f, 4.0f);
    CK(hipGetLastError());
    // outputs
    const size_t nQ = 2 * act_plane(cap, kD), nKV = (size_t)kCtx * kD, nH = 2 * act_plane(cap, kFp);
    uint16_t *Q = dev<uint16_t>(nQ, 0), *Kc = dev<uint16_t>(nKV, 0), *Vt = dev<uint16_t>(nKV, 0);
    uint16_t *H = dev<uint16_t>(nH, 0), *An = dev<uint16_t>(nAd, 0);
    float *X = dev<float>((size_t)cap * kD, 0), *ssq_out = dev<float>((size_t)(kD / 16) * cap, 0);
    float *part = dev<float>((size_t)kDownSplits * cap * kD, 0);
    float *spart = dev<float>((size_t)4 * cap * std::max(2 * kFp, kV), 0);
    float *sinv = dev<float>((size_t)cap, 0);
    const int n_wg_lm = (kV + 16 * kLmTiles - 1) / (16 * kLmTiles);
    float *pmax = dev<float>((size_t)n_wg_lm * cap, 0);
    int *pidx = dev<int>((size_t)n_wg_lm * cap, 0);

    struct Prod {
        const char *name;
        GemmKind kind;
        int cols, K;
    };
    const Prod prods[] = {{"qkv", GEMM_QKV, 3 * kD, kD}, {"o", GEMM_O, kD, kD}, {"gate_up", GEMM_GATE_UP, 2 * kFp, kD},
                          {"down", GEMM_DOWN, kD, kFp}, {"lm_head", GEMM_LM, n_wg_lm * 16 * kLmTiles, kD}};
    int bad = 0;
    for (int lt = 0; lt < 2; ++lt)
    for (const Prod &pr : prods) {
        if (lt == 1 && launch_tiles[1] == launch_tiles[0]) break;
        const int tiles_l = launch_tiles[lt];
        GemmParams p{};
        p.W = reinterpret_cast<const uint8_t *>(W);
        p.Ks = pr.K / 32;
        p.cols = pr.cols;
        p.A = pr.kind == GEMM_DOWN ? (const void *)A_f : (const void *)A_d;
        p.lda = pr.K;
        p.rr = RowsRef{tab, rinfo, cap};
        p.ssq = ssq;
        p.T = kD / 16;
        p.K = kD;
        p.eps = 1e-6f;
        p.Q = Q;
        p.Kc = Kc;
        p.Vt = Vt;
        p.kv_seq = 0;
        p.ctx_alloc = kCtx;
        p.rcos = rcos;
        p.rsin = rsin;
        p.d = kD;
        p.hd = kHd;
        p.Xout = X;
        p.ssq_out = ssq_out;
        p.ldx = kD;
        p.gain = gain;
        p.An = An;
        p.part = part;
        p.spart = spart;
        p.sinv = sinv;
        p.H = H;
        p.Fp = kFp;
        p.pmax = pmax;
        p.pidx = pidx;
        p.V = kV;
        std::vector<std::vector<uint16_t>> out16[2];
        std::vector<std::vector<float>> out32[2];
        std::vector<int> outi[2];
        for (int way = 0; way < 2; ++way) {
            CK(hipMemset(Q, 0, nQ * 2));
            CK(hipMemset(Kc, 0, nKV * 2));
            CK(hipMemset(Vt, 0, nKV * 2));
            CK(hipMemset(H, 0, nH * 2));
            CK(hipMemset(An, 0, nAd * 2));
            CK(hipMemset(ssq_out, 0, (size_t)(kD / 16) * cap * 4));
            CK(hipMemcpy(X, X0, (size_t)cap * kD * 4, hipMemcpyDeviceToDevice));
            CK(hipMemset(pmax, 0, (size_t)n_wg_lm * cap * 4));
            CK(hipMemset(pidx, 0, (size_t)n_wg_lm * cap * 4));
            GemmParams q = p;
            q.tile_kernel = way;  // 0: as iterations launch it, 1: gemm_kernel over the row tiles
            CK(launch_gemm(pr.kind, true, 4, tiles_l, q, 0, nullptr, nullptr));
            CK(hipDeviceSynchronize());
            out16[way] = {to_host(Q, nQ), to_host(Kc, nKV), to_host(Vt, nKV), to_host(H, nH), to_host(An, nAd)};
            out32[way] = {to_host(X, (size_t)cap * kD), to_host(ssq_out, (size_t)(kD / 16) * cap),
                          to_host(pmax, (size_t)n_wg_lm * cap)};
            outi[way] = to_host(pidx, (size_t)n_wg_lm * cap);
        }
        size_t d16 = 0, d32 = 0, n = 0;
        for (int i = 0; i < 5; ++i) {
            d16 += count_diff(out16[0][i], out16[1][i]);
            n += out16[0][i].size();
        }
        for (int i = 0; i < 3; ++i) {
            d32 += count_diff(out32[0][i], out32[1][i]);
            n += out32[0][i].size();
        }
        d32 += count_diff(outi[0], outi[1]);
        n += outi[0].size();
        std::printf("check %-8s rows=%d row_tiles=%d: %zu of %zu output values differ\n", pr.name, rows, tiles_l,
                    d16 + d32, n);
        bad += (d16 + d32) != 0;
    }
    std::printf(bad ? "check FAILED\n" : "check ok\n");
    return bad ? 1 : 0;
}
